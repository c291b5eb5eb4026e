// internal.h -- host-side structures and kernel launchers of libmnmt.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <map>
#include <string>
#include <vector>

#include "../../include/mnmt.h"

namespace mnmt {

// Status with message; set_error stores the thread-local text.
int set_error(int status, const std::string& msg);
int hip_error(hipError_t e, const char* what);

#define MNMT_HIP(call)                                      \
  do {                                                      \
    hipError_t _e = (call);                                 \
    if (_e != hipSuccess) return ::mnmt::hip_error(_e, #call); \
  } while (0)

// Epilogue kinds: the public MNMT_EPI_* values plus the fused arg-max.
enum : int { EPI_LOGITS_ARGMAX = 16 };

struct EpiArgs {
  int kind;
  void* out;          // [M, ldo] of the epilogue's type (may be null for ARGMAX)
  int ldo;            // row stride of out, in elements
  float gamma;        // residual weight for F32_RESID
  unsigned long long* argmax;  // [M] packed (value, ~index) maxima for ARGMAX
};

// Tiled matrix-core GEMM for large M (gemm.hip); K a multiple of 64.
// w4: W holds the packed 4-bit rows [N, K / 2] of the model file (16-code
// groups, byte i holding codes i and i + 8), widened to int8 on the way to
// the matrix cores.
hipError_t launch_gemm(const int8_t* X, int ldx, const int8_t* W, const float* scale, const float* bias, int M, int K,
                       int N, const EpiArgs& e, hipStream_t s, bool w4 = false);
// Y = epilogue(X[M,K] . W[N,K]^T); ldx = row stride of X in bytes; w4 as
// for launch_gemm (not with the fused arg-max).
hipError_t launch_qlinear(const int8_t* X, int ldx, const int8_t* W, const float* scale, const float* bias,
                          int M, int K, int N, const EpiArgs& e, hipStream_t s, bool w4 = false);

// LayerNorm (optional) + quantization of rows of x [rows, d]:
// do_ln: y = LN(x) with g, b, eps; else y = x.  q = quant(y, inv_s) if q;
// x_out = y if x_out (post-LN writes the normalized row back).
hipError_t launch_ln_quant(const float* x, int rows, int d, int do_ln, const float* g, const float* b, float eps,
                           float inv_s, int8_t* q, float* x_out, hipStream_t s);

// Token embedding + position table into x [rows, d]; row r of sentence
// (r / S) position p: encoder (tok = src[r], p = r % S); decoder
// (tok = tok[r], p = *step).
hipError_t launch_embed(const int32_t* tok, int rows, int S_for_pos, const int* step, const int8_t* E,
                        const float* c_emb, const float* pe, int d, int V, float* x, hipStream_t s);
// The same rows for a factorized embedding (Section 2.1): E [V, Ef] int8
// rows projected to d by P [d, Ef] (per-tensor scale s_proj):
// x = fma((float)(E[tok] . P[n]) * s_proj, c_emb[tok], PE[pos][n]).
constexpr int kMaxEmbDim = 1024;
hipError_t launch_embed_proj(const int32_t* tok, int rows, int S_for_pos, const int* step, const int8_t* E, int Ef,
                             const int8_t* P, float s_proj, const float* c_emb, const float* pe, int d, int V,
                             float* x, hipStream_t s);

// Encoder self-attention over qkv [B*S, 3d] -> ctx [B*S, d].
hipError_t launch_attn_enc(const int8_t* qkv, const int32_t* len, int B, int S, int d, int h, float c_qk,
                           float c_pv, int8_t* ctx, hipStream_t s);

// Decoder self-attention at position t (t_host when >= 0, the step index
// known when the work is enqueued, else *step): stores this step's k, v of every
// row into kcache/vcache [R][T][d] and attends over positions 0..step of the
// row's hypothesis (hist: two [R][T] tables, position -> cache row, the one
// of parity step & 1 is read; null = the row's own cache).
hipError_t launch_attn_dec_self(const int8_t* qkv, int R, int d, int h, int T, const int* step, int8_t* kcache,
                                int8_t* vcache, const int32_t* hist, float c_qk, float c_pv, int8_t* ctx,
                                hipStream_t s, int t_host = -1);

// The same with the Q/K/V projection inside (the batched decoder: one block
// per head and sentence of W <= 16 rows, d 128 or 256, heads 16-64 wide):
// rows are the int8 input rows [R, d], or with ln (rows null) the LayerNorm
// + quantization of ln->x computed by each block; wqkv [3d, d] (w4: packed
// 4-bit rows) with the I8 requantization of scale / bias.
struct FusedIn;
bool attn_self_qkv_fits(int W, int d, int h, int T);
hipError_t launch_attn_self_qkv(const int8_t* rows, const FusedIn* ln, const int8_t* wqkv, const float* scale,
                                const float* bias, bool w4, int R, int W, int d, int h, int T, const int* step,
                                int8_t* kcache, int8_t* vcache, const int32_t* hist, float c_qk, float c_pv,
                                int8_t* ctx, hipStream_t s, int t_host);

// Decoder cross-attention: row r attends over the cross keys/values of
// sentence r / W (kv [B*S, 2d]) limited to len[b].
hipError_t launch_attn_dec_cross(const int8_t* q, int R, int W, int d, int h, const int8_t* kv, int S,
                                 const int32_t* len, float c_qk, float c_pv, int8_t* ctx, hipStream_t s);

// The same with the query projection fused (the cross-attention's Q linear
// layer: int8 rows [R, d] of the LayerNorm'd input, wq [d, d] int8 or, w4,
// packed 4-bit, the I8 requantization with q_scale / q_bias), for W <= 16
// and d 256 (attn_cross_q_fits).
bool attn_cross_q_fits(int W, int d);
// rows: the int8 input rows [R, d], or with ln (rows null) the LayerNorm +
// quantization of ln->x computed by each block for its sentence's rows.
struct FusedIn;
hipError_t launch_attn_dec_cross_q(const int8_t* rows, const FusedIn* ln, const int8_t* wq, const float* q_scale,
                                   const float* q_bias, bool w4, int R, int W, int d, int h, const int8_t* kv, int S,
                                   const int32_t* len, float c_qk, float c_pv, int8_t* ctx, hipStream_t s);

// Greedy bookkeeping after the fused logits/arg-max of a step.
// out_key [T][R] (or null) receives each step's winning arg-max key.
hipError_t launch_greedy_commit(unsigned long long* slots, int R, int T, int32_t* cur_tok, int32_t* out_tok,
                                int32_t* finished, int32_t* out_len, int* step, int stop_at_eos, int eos,
                                int pad, unsigned long long* out_key, hipStream_t s);
// Also advances the counted hand-off's translation counter *epoch (if not null).
hipError_t launch_greedy_reset(unsigned long long* slots, int R, int steps, int32_t* cur_tok, int32_t* finished,
                               int32_t* out_len, int* step, int bos, unsigned long long* fslots, int n_fslots,
                               unsigned* epoch, hipStream_t s);
// A nonzero *chain_err (a chained kernel's wait gave up) marks every row's
// length -1 instead of copying it.
hipError_t launch_greedy_output(const int32_t* out_tok, const int32_t* out_len, int R, int T, int32_t* out,
                                int32_t* out_len_dst, const int* chain_err, hipStream_t s);
// The length penalties ((5 + L) / 6)^alpha, L = 0 .. n - 1, computed on the
// host and passed by value in the kernel's arguments, into dst [n].
struct LpTable {
  static constexpr int kMax = 257;  // max_tgt_len <= 256
  float v[kMax];
  int n;
};
hipError_t launch_fill_lp(const LpTable& tab, float* dst, hipStream_t s);
// Arg-max of fp32 rows [R, V] into packed slots (greedy when logits are
// produced by the matrix-core path).
hipError_t launch_row_argmax(const float* z, int R, int V, unsigned long long* slots, hipStream_t s);
// Copy tokens into/out of the session (int32 vectors).
hipError_t launch_load_batch(const int32_t* src_in, const int32_t* len_in, int32_t* src, int32_t* len, int n_src,
                             int n_len, unsigned* zero, int n_zero, hipStream_t s);
hipError_t launch_copy_i32(const int32_t* src, int32_t* dst, int n, hipStream_t s);
// Fragment order of an int8 weight [N, K] (K a multiple of 64) for the batch-1
// logits kernel: per tile t of 16 rows and slice j of 64 columns, one
// contiguous kilobyte whose 16-byte chunk l holds row 16t + l % 16, columns
// 64j + 16(l / 16) .. +15 (the i8 16x16x64 MFMA operand of lane l); rows past
// N are zero.  frag_bytes = ceil(N / 16) * 16 * K (0 for bad sizes).
size_t frag_bytes(int N, int K);
hipError_t launch_pack_fragments(const int8_t* W, int N, int K, int8_t* out, hipStream_t s);

// Fused decoder step for up to 8 rows (decode_fused.hip).
struct FusedIn {           // how a kernel obtains its int8 input rows
  const float* x;          // residual rows [R, d] (unused when embed)
  float* x_out;            // block 0 writes the input (wb_input) or normalized rows here, or null
  int wb_input;
  int embed;               // 1: rows are the embeddings of tok[] at position *step
  const int32_t* tok;
  const int8_t* E;
  const float* c_emb;
  const float* pe;
  int V;
  int S_pos;               // > 0: embedding position = row % S_pos (encoder); 0: the decode step
  int do_ln;               // LayerNorm before quantization
  const float* g;
  const float* b;
  float eps;
  float inv_s;             // 1 / input scale of the consuming linear layer
  // a pending residual update (nparts > 0): x <- fma(pgamma, x, fma(acc,
  // pscale, pbias)) with acc the sum of nparts int32 slices part + p
  // part_stride (a linear layer's partial sums over ranges of its K); the
  // writer blocks store the updated rows to x_out (wb_input)
  const int32_t* part;
  int nparts;
  size_t part_stride;
  const float* pscale;
  const float* pbias;
  float pgamma;
};
struct FusedGemv {         // a linear layer over the prepared rows, and greedy bookkeeping
  int R, K, N;
  int t;                   // decode step (position) of this launch
  int epi;                 // MNMT_EPI_I8, MNMT_EPI_I8_RELU or EPI_LOGITS_ARGMAX
  const int8_t* W;
  bool w4;                 // W holds packed 4-bit rows (K / 2 bytes each; not with the arg-max)
  const float* scale;
  const float* bias;
  void* out;               // int8 [R, N]; for the arg-max: fp32 logits [R, N] or null
  unsigned long long* slots;  // arg-max: [R][nslots], zero before the launch
  int nslots;              // arg-max slots per row (fused_slots_per_row(V))
  int* step;               // commit: advanced to t + 1
  int32_t* out_tok;
  int32_t* cur_tok;
  int32_t* finished;
  int32_t* out_len;
  unsigned long long* out_key;  // commit: [T][R] the step's winning arg-max key (or null)
  int T, stop_at_eos, eos, pad;
  int tagged;              // commit: the slots hold tagged keys (tagged_key)
  int32_t* zero_acc;       // commit: cleared after the step (or null)
  int zero_n;
  float* emb_out;          // commit: embedding of the next input tokens at position t + 1 (or null)
  const int8_t* E;
  const float* c_emb;
  const float* pe;
  int d, V, P;
};
hipError_t launch_qgemv_ln(const FusedIn& in, const FusedGemv& gv, hipStream_t s);

// Decoder step in 3 kernels per layer for at most 2 rows (decode_step.hip).
// Hand-off between consecutive kernels of a batch-1 translation that run on
// two alternating streams: a kernel loads its weights, then waits until every
// block of the kernel before it has stored `want` (or more) into its flag
// word, and its own blocks store `val` when done (release / acquire at agent
// scope).  Null `wait` / `done`: no wait / no flag.  Waits are bounded: after
// kChainSpinLimit polls the kernel sets *err and goes on.
// A kernel of at most kChainCopyStride blocks stores its flag words in
// kChainCopies copies kChainCopyStride words apart, and consumer block b
// polls copy b mod kChainCopies: hundreds of blocks polling one cache line
// serialize at the memory and delay everything around them.
constexpr int kChainMaxBlocks = 256;   // blocks of one kernel of the chain
constexpr int kChainCopies = 8, kChainCopyStride = 128;
constexpr int kChainSlotWords = kChainCopies * kChainCopyStride;  // flag words per kernel slot
constexpr unsigned kChainSpinLimit = 1u << 17;  // about 8 ms of polling
__host__ __device__ constexpr int chain_copies(int blocks) { return blocks <= kChainCopyStride ? kChainCopies : 1; }
struct StepChain {
  const unsigned* wait;  // the previous kernel's flag words [nwait]
  int nwait;
  unsigned want;
  unsigned* done;        // this kernel's flag words [gridDim.x]
  unsigned val;
  int* err;
};

// Counted hand-off between consecutive step kernels (instead of flags):
// the int32 partial sums of a kernel's blocks are added into 64-bit words,
// the sum modulo 2^32 in the low half and one count of 2^40 per adding block
// (at most 255 blocks: the low half's carries stay below bit 40), so a
// consumer polls the very words it needs until their count equals the
// producer's block count; block 0 of the producer stores its updated fp32
// rows as 64-bit words tagged with (translation, step, kernel).  The
// producer needs no wait for its atomics and no flag, the consumer no cache
// invalidation and no second load.
constexpr unsigned kTagSpan = 8192;  // row tag = epoch * kTagSpan + step * 32 + kernel index in the step
constexpr unsigned long long kCountUnit = 1ull << 40;
struct StepCount {
  int count_in;                       // > 0: poll acc until this many blocks added, rows from x_in64
  const unsigned long long* x_in64;   // [R][d] the previous kernel's tagged rows
  unsigned tag_in;                    // their tag offset
  unsigned long long* x_out64;        // [R][d] this kernel's rows, tagged (block 0), or null
  unsigned tag_out;
  const unsigned* epoch;              // translation counter (advanced by each reset)
};

struct StepIn {            // the sublayer input rows of a step kernel
  // Every pointer is valid for the extent given even where its flag is off,
  // so that the kernels load without branches.
  const float* x_in;       // residual rows [R, d]
  float* x_out;            // block 0 stores the updated rows here (or null)
  const unsigned long long* acc;  // [R, d] counted sums (StepCount): pending x <- fma(gamma, x, fma(acc, scale, bias))
  const float* scale;      // [d]
  const float* bias;       // [d]
  float gamma;
  int update;              // apply the pending update
  const float* ln_g;       // [d] LayerNorm gain and bias
  const float* ln_b;
  int ln_mode;             // 0 none, 1 post-LN (the residual stream), 2 pre-LN (the sublayer input)
  float eps;
  float inv_s;             // 1 / input scale of the consuming layer
  unsigned long long* zero_acc;  // block 0 clears this accumulator (its consumer has finished)
  int zero_n;
  StepChain chain;
  StepCount cnt;
};
struct StepAttn {
  int R, d, dh, T, S, t;
  const int8_t* W;         // QKV [3d, d] (self) or Q [d, d] (cross)
  const float* scale;
  const float* bias;
  const int8_t* Wo;        // output projection [d, d]
  int8_t* kcache;
  int8_t* vcache;
  const int8_t* kv;        // cross keys|values [R][S][2d]
  const int32_t* len;
  float c_qk, c_pv;
  unsigned long long* acc_out;  // [R, d] counted sums (StepCount), zero on entry
  bool w4;                 // W and Wo hold packed 4-bit rows (K / 2 bytes each)
};
// The greedy commit of the previous step's token, folded into the next
// step's first layer: the self-attention kernel of layer 0 reads the previous
// logits kernel's per-block arg-max partials and embeds the token itself (at
// position t), and block 0 of the cross-attention kernel of layer 0 records it
// (the bookkeeping runs one kernel later, so no block reads `finished` while
// another writes it).
struct StepCommit {
  const unsigned long long* slots;  // [R][nslots] arg-max partials of step t - 1
  int nslots;                       // at most 256
  int tagged;                       // partials are tagged keys (tagged_key), polled until all carry step t - 1's tag
  int nparts;                       // tagged: partials written per row (one per logits block)
  const unsigned* epoch;            // tagged: the translation counter of the tags
  const int8_t* E;                  // embedding [V, d], its scales, the position table
  const float* c_emb;
  const float* pe;
  int V;
  int t;                            // this step (the committed token is step t - 1's)
  int32_t* finished;
  int32_t* out_tok;                 // [T][R]
  int32_t* out_len;
  int32_t* cur_tok;
  unsigned long long* out_key;      // [T][R] the winning arg-max key of each step (or null)
  int* step;
  int T, stop_at_eos, eos, pad;
};
struct StepFfn {
  int R, d, F;
  const int8_t* W1;
  const float* scale1;
  const float* bias1;
  const int8_t* W2;        // [d, F]
  unsigned long long* acc_out;  // [R, d] counted sums (StepCount)
  bool w4;                 // W1 and W2 hold packed 4-bit rows
};
struct StepLogits {
  int R, d, V;
  const int8_t* E;
  const float* c_out;
  float* logits;           // [R, V] or null
  unsigned long long* slots;
  int nslots;
  const int8_t* x_i8;      // int8 rows [R, d] instead of the StepIn rows (or null)
  bool frag;               // E in fragment order (launch_pack_fragments), else row-major [V, d]
  int tagged;              // store tagged keys (tagged_key) for step t; V <= kTagMaxV
  const unsigned* epoch;
  int t;
};
// Tagged arg-max keys: the ordered value in bits 63..32, a 14-bit tag of the
// (translation, step) in bits 31..18 and 0x3FFFF - index in bits 17..0, so
// that among keys of one tag the maximum is still the arg max with the
// smallest index; a partial whose tag is the step's own is that step's.
// Tags run 1..16383 and never 0, the tag of a cleared slot: with tag 0 in
// use (the old & 0x3FFF form), every 64th translation's second step took the
// cleared slots for the first step's partials.
constexpr int kTagMaxV = 1 << 18;
__host__ __device__ inline unsigned step_tag(unsigned epoch, int t) {
  return 1u + (epoch * 256u + (unsigned)t) % 0x3FFFu;
}
bool step_path_fits(int R, int d, int dh, int F, int T, int S);
bool step_logits_fits(int R, int d);  // R <= 2, d a multiple of 64 up to 512
int step_logits_blocks(int V);        // blocks (and arg-max partials per row) of launch_step_logits
int step_logits_blocks_chained(int V, int d);  // the same in a kernel chain (more rows per block)
// cm (or null): self = 1 embeds the previous step's token from its partials
// (layer 0, the rows' x_in unused); self = 0 records that token (block 0).
hipError_t launch_step_attn(const StepIn& in, const StepAttn& at, int self, int heads, hipStream_t s,
                            const StepCommit* cm = nullptr);
hipError_t launch_step_ffn(const StepIn& in, const StepFfn& f, hipStream_t s);
// One whole decoder layer (self attention, cross attention, FFN) in one
// launch of step_layer_blocks(heads, F) blocks, the phases handing off through
// the counted words (ib and ic take counted input); cm: the folded commit of
// the first layer (as launch_step_attn).  ic.chain carries the launch's flags.
int step_layer_blocks(int heads, int F);
hipError_t launch_step_layer(const StepIn& ia, const StepAttn& sa, const StepIn& ib, const StepAttn& ca,
                             const StepIn& ic, const StepFfn& f, hipStream_t s, const StepCommit* cm = nullptr);
// The whole step of a two-layer decoder in one launch (k_step_all): the two
// layers' role arguments as launch_step_layer takes them, the first layer's
// folded commit, and the logits kernel's arguments (chained form: its input
// waits on the last layer's flags).
struct StepAll {
  StepIn ia[2], ib[2], ic[2];
  StepAttn sa[2], ca[2];
  StepFfn f[2];
  StepCommit cm;
  StepIn lin;
  StepLogits g;
  int layer_blocks;  // step_layer_blocks(heads, F)
};
// Whether k_step_all covers a step: two layers of width 256, at
// most 64 attended positions (self and cross), a vocabulary the tagged
// logits take with 4 tiles of 16 rows per wave (V >= 24576).
bool step_all_fits(int n_dec, int d, int heads, int F, int T, int S, int V);
hipError_t launch_step_all(const StepAll& p, bool fold, hipStream_t s);
// With ev_start / ev_stop the events take the kernel's own start and end times.
hipError_t launch_step_logits(const StepIn& in, const StepLogits& g, hipStream_t s, hipEvent_t ev_start = nullptr,
                              hipEvent_t ev_stop = nullptr);
// Encoder for at most 64 rows in 2 kernels per layer (encode_small.hip).
struct EncIn {             // the sublayer input rows of an encoder kernel
  // Every pointer is valid for the extent given even where its flag is off.
  int R, d, S;             // rows (B * S), width, positions per sentence
  int embed;               // rows = embeddings of tok[r] at position r % S
  const int32_t* tok;
  const int8_t* E;
  const float* c_emb;
  const float* pe;
  int V;
  const float* x_in;       // residual rows [R, d]
  float* x_out;            // the blocks store the updated rows here (or null)
  const int32_t* acc;      // [R, d]: pending update x <- fma(gamma, x, fma(acc, scale, bias))
  const float* scale;      // [d]
  const float* bias;       // [d]
  float gamma;
  int update;
  const float* ln_g;       // [d]
  const float* ln_b;
  int ln_mode;             // 0 none, 1 post-LN (the residual stream), 2 pre-LN (the sublayer input)
  float eps;
  float inv_s;             // 1 / input scale of the consuming layer
  int8_t* q_out;           // the blocks store the int8 rows here (or null)
  int32_t* zero0;          // the blocks clear these accumulators (their consumers have finished);
                           // zero0_n, zero1_n: multiples of 64
  int nblk;                // blocks of the launch (set by the launcher)
  int zero0_n;
  int32_t* zero1;
  int zero1_n;
  StepChain chain;
};
struct EncAttn {
  int dh;
  const int8_t* W;         // QKV [3d, d]
  const float* scale;
  const float* bias;
  const int8_t* Wo;        // [d, d]
  const int32_t* len;      // [B]
  float c_qk, c_pv;
  int32_t* acc_out;        // [R, d], zero on entry
  int qsplit;              // blocks per head (set by the launcher): each takes every qsplit-th 16-row query tile
  bool w4;                 // W and Wo hold packed 4-bit rows
};
struct EncFfn {
  int F;
  const int8_t* W1;
  const float* scale1;
  const float* bias1;
  const int8_t* W2;        // [d, F]
  int32_t* acc_out;        // [R, d], zero on entry
  bool w4;                 // W1 and W2 hold packed 4-bit rows
};
struct EncOut {            // every decoder layer's cross K|V projection of the encoder output
  static constexpr int kMaxLayers = 16;
  struct Layer {
    const int8_t* W;       // [2d, d]
    const float* scale;
    const float* bias;
    int8_t* out;           // [R, 2d]
  } layer[kMaxLayers];
  int layers;
  bool w4;                 // every layer's W holds packed 4-bit rows
};
bool enc_small_fits(int R, int S, int d, int dh, int F);
int enc_attn_qsplit(int R);  // blocks per head of launch_enc_attn for R rows
hipError_t launch_enc_attn(const EncIn& in, const EncAttn& at, int heads, hipStream_t s);
hipError_t launch_enc_ffn(const EncIn& in, const EncFfn& f, hipStream_t s);
hipError_t launch_enc_out(const EncIn& in, const EncOut& o, hipStream_t s);

// Small-M GEMM (M <= 64, K <= 1024; up to 512 rows for the shapes
// qgemm_rows_fit accepts) on 16x16x64 matrix cores; with `in` the rows are
// prepared (embedding / LayerNorm / quantization, rows up to 1024 wide) in
// its prologue.
bool qgemm_small_fits(int M, int K);
bool qgemm_rows_fit(int M, int K, int N);
hipError_t launch_qgemm_small(const FusedIn* in, const int8_t* X, int ldx, const int8_t* W, const float* scale,
                              const float* bias, int M, int K, int N, const EpiArgs& e, hipStream_t s,
                              bool w4 = false);
// Long-K linear layers of the batched decoder (the feed-forward W2 of wide
// models): K split into kSplitKb-column ranges, one row of the tiled GEMM's
// grid each,
// whose int32 partial sums go to part [splits][M][N]; the next row kernel
// (launch_resid_ln_quant) adds them (integer sums: exact in any order) and
// applies the residual epilogue.  qgemm_splits: the split count for a shape,
// 0 where the split does not apply (it needs 8 < M <= 512, N <= 1024, K a
// multiple of kSplitKb above 1024 with at most kMaxSplits ranges: shorter K
// takes the one-round-trip kernel whole).
constexpr int kSplitKb = 512, kMaxSplits = 4;
int qgemm_splits(int M, int K, int N);
hipError_t launch_qgemm_split(const int8_t* X, int ldx, const int8_t* W, int M, int K, int N, int32_t* part,
                              hipStream_t s, bool w4 = false);
// The tiled GEMM's K split behind it (64x64 tiles, `splits` K ranges).
hipError_t launch_gemm_split(const int8_t* X, int ldx, const int8_t* W, int M, int K, int N, int splits,
                             int32_t* part, hipStream_t s, bool w4);
// A residual update pending from a linear layer's int32 sums:
// x <- fma(gamma, x, fma((float)(sum of the splits' partials), scale, bias)),
// the expression of the MNMT_EPI_F32_RESID epilogue.
struct ResidUpdate {
  const int32_t* part;  // [splits][rows][d]
  int splits;
  const float* scale;
  const float* bias;
  float gamma;
};
// launch_ln_quant after the pending update of the rows x [rows, d], which are
// stored back (pre-LN: the updated rows; post-LN: x_out = x, the normalized
// rows replace them).
hipError_t launch_resid_ln_quant(float* x, int rows, int d, const ResidUpdate& u, int do_ln, const float* g,
                                 const float* b, float eps, float inv_s, int8_t* q, bool post, hipStream_t s);
hipError_t launch_greedy_commit_slots(const FusedGemv& gv, hipStream_t s);
// Arg-max slots per row of the greedy paths: the spread atomic slots of the
// 3-8 row path and one partial per block of the 1-2 row logits kernel.
int fused_slots_per_row(int V);

// Beam search kernels.
struct BeamState {
  int B, W, V, T;
  float* score;          // [R] live scores
  float* cand_score;     // [R][2W] per-row best expansions
  int32_t* cand_tok;     // [R][2W]
  int32_t* tok_hist;     // [T][R] token chosen into slot r at step t
  int32_t* par_hist;     // [T][R] parent row of slot r at step t
  int32_t* hist;         // [2][R][T] position -> cache row, double buffered by step parity
  float* fin_score;      // [B][W]
  int32_t* fin_len;      // [B][W]
  int32_t* fin_row;      // [B][W] row of the EOS candidate's parent (hypothesis) at step len-1
  int32_t* fin_count;    // [B]
  int32_t* done;         // [B]
  int32_t* cur_tok;      // [R]
  const float* lp;       // [T + 1] length penalties
  int32_t* count;        // [1] blocks of the update kernel finished this step (0 between steps)
  int eos, pad, bos;
  int t_host = -1;       // >= 0: the step index, known when the work is enqueued (else the kernels read *step)
};
// The next step's input rows, written by the beam update for every slot of
// its sentence while t + 1 < steps: the embedding of the slot's token at
// position t + 1 (x) and the first decoder layer's int8 input (a: LayerNorm
// when do_ln, then quantization with inv_s).
struct BeamNext {
  float* x;        // [R, d]
  int8_t* a;       // [R, d]
  const int8_t* E;
  const float* c_emb;
  const float* pe;  // [P, d]
  int d, V, P, steps;
  int do_ln;
  const float* g;
  const float* b;
  float eps, inv_s;
};
hipError_t launch_beam_reset(const BeamState& st, int* step, hipStream_t s);
hipError_t launch_beam_topk(const float* logits, const BeamState& st, const int* step, hipStream_t s);
// Also advances the step counter (the last block to finish).
hipError_t launch_beam_update(const BeamState& st, int* step, const BeamNext& nx, hipStream_t s);
// A nonzero *chain_err marks every sentence's length -1 (see launch_greedy_output).
hipError_t launch_beam_finalize(const BeamState& st, int steps, int32_t* out, int32_t* out_len, float* out_score,
                                const int* chain_err, hipStream_t s);

// Model files (model.cpp); flags: MNMT_LOAD_* of mnmt.h.
int model_size(const void* blob, size_t n, unsigned flags, size_t* bytes, std::string& err);
int model_create(const void* blob, size_t n, unsigned flags, void* d_arena, size_t arena_bytes, hipStream_t s,
                 mnmt_model** out, std::string& err);

// Canonical-arithmetic self check.
hipError_t launch_debug_canon(int fn, const float* x, int n, float* y, hipStream_t s);
// Read bandwidth probe: kDebugReadBlocks blocks read `bytes` (a multiple of
// 16) `reps` times, each block the same share every time, and each stores one
// word of sink [kDebugReadBlocks].
constexpr int kDebugReadBlocks = 2048;
hipError_t launch_debug_read(const void* x, size_t bytes, int reps, unsigned* sink, hipStream_t s);

// ---------------------------------------------------------------------------
// Model and session structures.

struct LinearDev {
  const int8_t* w = nullptr;    // [N, K] int8 codes (null: 4-bit weights loaded packed only)
  const uint8_t* w4 = nullptr;  // 4-bit weights: the packed rows [N, K / 2] of the model file, else null
  const float* scale = nullptr;
  const float* bias = nullptr;
  int N = 0, K = 0;
  float inv_in = 0.f;  // 1 / input scale (quantization of this layer's input)
};

// The weight a batched kernel reads: the int8 codes, or the packed 4-bit
// rows when the model keeps only those (returns true).
inline bool batched_weights(const LinearDev& a, const int8_t*& w) {
  w = a.w ? a.w : reinterpret_cast<const int8_t*>(a.w4);
  return a.w == nullptr;
}

// A 1-2 row kernel's pair of weights: the packed 4-bit rows when both have
// them (returns true), else the int8 codes.
inline bool pick_weights(const LinearDev& a, const LinearDev& b, const int8_t*& wa, const int8_t*& wb) {
  if (a.w4 && b.w4) {
    wa = reinterpret_cast<const int8_t*>(a.w4);
    wb = reinterpret_cast<const int8_t*>(b.w4);
    return true;
  }
  wa = a.w;
  wb = b.w;
  return false;
}

struct LnDev {
  const float* g = nullptr;
  const float* b = nullptr;
};

struct LayerDev {
  LnDev sa_ln, ca_ln, ff_ln;
  LinearDev qkv, o, cq, ckv, co, w1, w2;
  float sa_gamma = 1.f, ca_gamma = 1.f, ff_gamma = 1.f;
  float sa_cqk = 0.f, sa_cpv = 0.f, ca_cqk = 0.f, ca_cpv = 0.f;
};

}  // namespace mnmt

struct mnmt_model {
  mnmt_model_info info{};
  int dh = 0;
  int device = 0;
  size_t arena_bytes = 0;
  const int8_t* E = nullptr;     // [V, d]
  const int8_t* E_frag = nullptr;  // E in fragment order, frag_bytes(V, d) (the batch-1 logits)
  const float* c_emb = nullptr;  // [V]
  const float* c_out = nullptr;  // [V]
  const float* pe = nullptr;     // [P, d]
  bool packed_only = false;      // 4-bit weights without their int8 copies (MNMT_LOAD_PACKED_4BIT_ONLY)
  // factorized embedding (info.emb_dim > 0): E is [V, emb_dim], proj [d,
  // emb_dim] maps it to the model width, proj_out (its transpose, requantized
  // with s_fin * s_proj / s_u) maps the final rows back to emb_dim
  const int8_t* proj = nullptr;
  float s_proj = 0.f;
  mnmt::LinearDev proj_out;
  std::vector<mnmt::LayerDev> enc, dec;
  std::vector<int> enc_alias, dec_alias;  // layer l reuses layer alias[l]'s parameters (-1: its own)
  mnmt::LnDev enc_ln, dec_ln;
  float s_enc = 0.f, inv_enc = 0.f, inv_fin = 0.f;
};

struct mnmt_session {
  const mnmt_model* m = nullptr;
  mnmt_session_cfg cfg{};
  int R = 0;  // max rows = max_batch * beam
  // current batch
  int B = 0, S = 0, W = 1;
  bool encoded = false;
  int host_step = 0;
  // buffers (device)
  int32_t* src = nullptr;
  int32_t* len = nullptr;
  float* enc_x = nullptr;
  int8_t* enc_a = nullptr;
  int8_t* enc_qkv = nullptr;
  int8_t* enc_h = nullptr;
  int8_t* enc_out = nullptr;
  float* enc_x2 = nullptr;  // second encoder residual buffer (post-LN ping-pong)
  float* logits = nullptr;  // shares memory with the encoder scratch
  std::vector<int8_t*> cross_kv;
  float* dec_x = nullptr;
  float* dec_x2 = nullptr;  // second residual buffer (post-LN ping-pong)
  unsigned long long* fslots = nullptr;  // arg-max slots [8][fused_slots_per_row(V)]
  unsigned long long* step_acc = nullptr;  // decode-step accumulators [3][2][d], counted 64-bit words
  int32_t* enc_acc = nullptr;            // small-batch encoder accumulators [2 W_o + 2 W2][64][d] int32
  int8_t* dec_a = nullptr;
  int8_t* dec_qkv = nullptr;
  int8_t* dec_q = nullptr;
  int8_t* dec_h = nullptr;
  int8_t* dec_u = nullptr;  // factorized embedding: the output projection's int8 input [R, emb_dim]
  int32_t* dec_part = nullptr;  // split-K partial sums [kMaxSplits][R][d] (launch_qgemm_split)
  std::vector<int8_t*> kcache, vcache;
  int32_t* cur_tok = nullptr;
  int* step = nullptr;
  unsigned long long* slots = nullptr;
  int32_t* out_tok = nullptr;
  int32_t* finished = nullptr;
  int32_t* out_len = nullptr;
  unsigned long long* out_key = nullptr;  // [T][R] greedy: each step's winning arg-max key
  float* lp = nullptr;
  mnmt::BeamState beam{};
  std::map<std::string, std::pair<void*, size_t>> named;
  // graph cache
  hipStream_t capture_stream = nullptr;
  hipStream_t side_stream = nullptr;  // the second stream of the batch-1 kernel chain
  hipEvent_t fork_ev = nullptr, join_ev = nullptr;
  unsigned* chain = nullptr;          // flag words [3 n_dec + 1][kChainSlotWords], cleared per translation
  unsigned* enc_chain = nullptr;      // the encoder's [2 n_enc][kChainSlotWords], cleared by the batch load
  int* chain_err = nullptr;           // set by a wait that gave up (cleared by mnmt_session_status)
  unsigned* epoch = nullptr;          // translation counter of the counted hand-off's row tags
  unsigned long long* step_x64 = nullptr;  // tagged rows of the step kernels [3 n_dec][2][d]
  bool counted_on = true;             // off with MNMT_COUNTED=0: flags between all step kernels
  bool merged_on = true;              // off with MNMT_MERGED_LAYERS=0: three launches per decoder layer
  bool tagged_on = true;              // off with MNMT_TAGGED=0: layer 0 waits on the logits kernel's flags
  bool single_on = false;             // on with MNMT_STEP_LAUNCH=1: one launch per step (k_step_all)
  bool ln_fused_on = true;            // off with MNMT_LN_FUSED=0: batched LayerNorms as kernels of their own
  bool qkv_fused_on = true;           // off with MNMT_QKV_FUSED=0: the batched Q/K/V projection as its own GEMM
  bool chain_on = true;               // off with MNMT_SERIAL_STEPS=1 in the environment
  std::map<std::string, hipGraphExec_t> graphs;
};
