// api.cpp -- C ABI entry points for models, single linear layers, the
// canonical-arithmetic self check and error reporting.
#include <cmath>
#include <string>

#include "internal.h"

namespace mnmt {

namespace {
thread_local std::string g_last_error;
}

int set_error(int status, const std::string& msg) {
  g_last_error = msg;
  return status;
}

int hip_error(hipError_t e, const char* what) {
  return set_error(MNMT_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

}  // namespace mnmt

using namespace mnmt;

extern "C" const char* mnmt_status_str(int status) {
  switch (status) {
    case MNMT_OK: return "ok";
    case MNMT_E_INVALID_ARG: return "invalid argument";
    case MNMT_E_BAD_MODEL: return "bad model file";
    case MNMT_E_CAPACITY: return "capacity exceeded";
    case MNMT_E_HIP: return "HIP runtime error";
    case MNMT_E_UNSUPPORTED: return "unsupported";
    case MNMT_E_TIMEOUT: return "device-side wait timed out";
    default: return "unknown status";
  }
}

extern "C" const char* mnmt_last_error(void) { return g_last_error.c_str(); }

extern "C" int mnmt_model_bytes_ex(const void* blob, size_t blob_bytes, unsigned flags, size_t* device_bytes) {
  if (!device_bytes) return set_error(MNMT_E_INVALID_ARG, "device_bytes is null");
  std::string err;
  const int rc = model_size(blob, blob_bytes, flags, device_bytes, err);
  return rc ? set_error(rc, err) : MNMT_OK;
}

extern "C" int mnmt_model_bytes(const void* blob, size_t blob_bytes, size_t* device_bytes) {
  return mnmt_model_bytes_ex(blob, blob_bytes, 0u, device_bytes);
}

extern "C" int mnmt_model_load_ex(const void* blob, size_t blob_bytes, unsigned flags, void* d_arena,
                                  size_t arena_bytes, void* stream, mnmt_model** out) {
  if (!out || !d_arena) return set_error(MNMT_E_INVALID_ARG, "out or arena is null");
  std::string err;
  const int rc =
      model_create(blob, blob_bytes, flags, d_arena, arena_bytes, static_cast<hipStream_t>(stream), out, err);
  return rc ? set_error(rc, err) : MNMT_OK;
}

extern "C" int mnmt_model_load(const void* blob, size_t blob_bytes, void* d_arena, size_t arena_bytes, void* stream,
                               mnmt_model** out) {
  return mnmt_model_load_ex(blob, blob_bytes, 0u, d_arena, arena_bytes, stream, out);
}

extern "C" int mnmt_model_get_info(const mnmt_model* model, mnmt_model_info* out) {
  if (!model || !out) return set_error(MNMT_E_INVALID_ARG, "null argument");
  *out = model->info;
  return MNMT_OK;
}

extern "C" void mnmt_model_free(mnmt_model* model) { delete model; }

extern "C" int mnmt_qlinear_timed(const int8_t* d_X, const int8_t* d_W, const float* d_scale, const float* d_bias,
                                  int M, int K, int N, int epilogue, float gamma, void* d_Y, void* stream,
                                  void* ev_start, void* ev_stop);

extern "C" int mnmt_qlinear(const int8_t* d_X, const int8_t* d_W, const float* d_scale, const float* d_bias, int M,
                            int K, int N, int epilogue, float gamma, void* d_Y, void* stream) {
  return mnmt_qlinear_timed(d_X, d_W, d_scale, d_bias, M, K, N, epilogue, gamma, d_Y, stream, nullptr, nullptr);
}

extern "C" int mnmt_qlinear_timed(const int8_t* d_X, const int8_t* d_W, const float* d_scale, const float* d_bias,
                                  int M, int K, int N, int epilogue, float gamma, void* d_Y, void* stream,
                                  void* ev_start, void* ev_stop) {
  if (M < 0 || N < 1 || K < 64 || K % 64 || K > 8192)
    return set_error(MNMT_E_INVALID_ARG, "need M >= 0, N >= 1 and K a multiple of 64 in [64, 8192]");
  if (epilogue < MNMT_EPI_I32 || epilogue > MNMT_EPI_ARGMAX_PARTIAL_PACKED)
    return set_error(MNMT_E_INVALID_ARG, "unknown epilogue");
  const bool packed = epilogue == MNMT_EPI_ARGMAX_PARTIAL_PACKED;
  if ((epilogue == MNMT_EPI_ARGMAX_PARTIAL || packed) && !step_logits_fits(M == 0 ? 1 : M, K))
    return set_error(MNMT_E_UNSUPPORTED, "the partial arg-max epilogue takes M <= 2 and K a multiple of 64 up to 512");
  if (epilogue == MNMT_EPI_ARGMAX && M > 8)
    return set_error(MNMT_E_UNSUPPORTED, "the fused arg-max epilogue takes at most 8 rows");
  if (M == 0) return MNMT_OK;
  const bool needs_scale = epilogue != MNMT_EPI_I32;
  const bool argmax = epilogue == MNMT_EPI_ARGMAX || epilogue == MNMT_EPI_ARGMAX_PARTIAL || packed;
  const bool needs_bias = epilogue != MNMT_EPI_I32 && epilogue != MNMT_EPI_LOGITS && !argmax;
  if (!d_X || !d_W || !d_Y || (needs_scale && !d_scale) || (needs_bias && !d_bias))
    return set_error(MNMT_E_INVALID_ARG, "null device pointer");
  if (reinterpret_cast<uintptr_t>(d_X) % 16 || reinterpret_cast<uintptr_t>(d_W) % 16)
    return set_error(MNMT_E_INVALID_ARG, "X and W must be 16-byte aligned");
  if (argmax && step_logits_fits(M, K)) {
    // the decoder's fused logits + arg-max kernel on int8 rows: one slot per
    // row (atomics), or one partial per block and row (plain stores)
    StepLogits g{};
    g.R = M;
    g.d = K;
    g.V = N;
    g.E = static_cast<const int8_t*>(d_W);
    g.frag = packed;
    g.c_out = d_scale;
    g.slots = static_cast<unsigned long long*>(d_Y);
    g.nslots = epilogue == MNMT_EPI_ARGMAX ? 1 : step_logits_blocks(N);
    g.x_i8 = static_cast<const int8_t*>(d_X);
    const hipError_t h = launch_step_logits(StepIn{}, g, static_cast<hipStream_t>(stream),
                                            static_cast<hipEvent_t>(ev_start), static_cast<hipEvent_t>(ev_stop));
    return h == hipSuccess ? MNMT_OK : hip_error(h, "qlinear launch");
  }
  const hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t h = ev_start ? hipEventRecord(static_cast<hipEvent_t>(ev_start), s) : hipSuccess;
  if (h != hipSuccess) return hip_error(h, "qlinear start event");
  EpiArgs e{epilogue, d_Y, N, gamma, nullptr};
  if (epilogue == MNMT_EPI_ARGMAX) e = EpiArgs{EPI_LOGITS_ARGMAX, nullptr, N, 1.f, static_cast<unsigned long long*>(d_Y)};
  h = launch_qlinear(d_X, K, d_W, d_scale, d_bias, M, K, N, e, s);
  if (h != hipSuccess) return hip_error(h, "qlinear launch");
  h = ev_stop ? hipEventRecord(static_cast<hipEvent_t>(ev_stop), s) : hipSuccess;
  return h == hipSuccess ? MNMT_OK : hip_error(h, "qlinear stop event");
}

extern "C" int mnmt_qlinear_w4(const int8_t* d_X, const uint8_t* d_W4, const float* d_scale, const float* d_bias,
                               int M, int K, int N, int epilogue, float gamma, void* d_Y, void* stream) {
  if (M < 0 || N < 1 || K < 64 || K % 64 || K > 8192)
    return set_error(MNMT_E_INVALID_ARG, "need M >= 0, N >= 1 and K a multiple of 64 in [64, 8192]");
  if (epilogue < MNMT_EPI_I32 || epilogue > MNMT_EPI_ARGMAX_PARTIAL_PACKED)
    return set_error(MNMT_E_INVALID_ARG, "unknown epilogue");
  if (epilogue > MNMT_EPI_LOGITS)
    return set_error(MNMT_E_UNSUPPORTED, "4-bit weights take the epilogues MNMT_EPI_I32 .. MNMT_EPI_LOGITS");
  if (M == 0) return MNMT_OK;
  const bool needs_bias = epilogue != MNMT_EPI_I32 && epilogue != MNMT_EPI_LOGITS;
  if (!d_X || !d_W4 || !d_Y || (epilogue != MNMT_EPI_I32 && !d_scale) || (needs_bias && !d_bias))
    return set_error(MNMT_E_INVALID_ARG, "null device pointer");
  if (reinterpret_cast<uintptr_t>(d_X) % 16 || reinterpret_cast<uintptr_t>(d_W4) % 8)
    return set_error(MNMT_E_INVALID_ARG, "X must be 16-byte and W4 8-byte aligned");
  const EpiArgs e{epilogue, d_Y, N, gamma, nullptr};
  const hipError_t h = launch_qlinear(d_X, K, reinterpret_cast<const int8_t*>(d_W4), d_scale, d_bias, M, K, N, e,
                                      static_cast<hipStream_t>(stream), true);
  return h == hipSuccess ? MNMT_OK : hip_error(h, "qlinear launch");
}

extern "C" int mnmt_argmax_partials(int N) { return N < 1 ? -1 : step_logits_blocks(N); }

extern "C" size_t mnmt_packed_bytes(int N, int K) { return frag_bytes(N, K); }

extern "C" int mnmt_pack_weights(const int8_t* d_W, int N, int K, int8_t* d_P, void* stream) {
  if (!frag_bytes(N, K)) return set_error(MNMT_E_INVALID_ARG, "need N >= 1 and K a positive multiple of 64");
  if (!d_W || !d_P) return set_error(MNMT_E_INVALID_ARG, "null device pointer");
  if (reinterpret_cast<uintptr_t>(d_W) % 16 || reinterpret_cast<uintptr_t>(d_P) % 16)
    return set_error(MNMT_E_INVALID_ARG, "W and P must be 16-byte aligned");
  const hipError_t h = launch_pack_fragments(d_W, N, K, d_P, static_cast<hipStream_t>(stream));
  return h == hipSuccess ? MNMT_OK : hip_error(h, "pack launch");
}

extern "C" int mnmt_fold_requant(float s_in, const float* s_w, const float* b, float s_out, int N, float* scale,
                                 float* bias) {
  if (!s_w || !b || !scale || !bias || N < 1 || !(s_in > 0.0f) || !(s_out > 0.0f))
    return set_error(MNMT_E_INVALID_ARG, "bad fold_requant arguments");
  for (int n = 0; n < N; ++n) {
    scale[n] = (float)((double)s_in * (double)s_w[n] / (double)s_out);
    bias[n] = (float)((double)b[n] / (double)s_out);
  }
  return MNMT_OK;
}

extern "C" int mnmt_debug_canon(int fn, const float* d_x, int n, float* d_y, void* stream) {
  if (fn < 0 || fn > 2 || n < 0 || !d_x || !d_y) return set_error(MNMT_E_INVALID_ARG, "bad debug_canon arguments");
  const hipError_t h = launch_debug_canon(fn, d_x, n, d_y, static_cast<hipStream_t>(stream));
  return h == hipSuccess ? MNMT_OK : hip_error(h, "debug_canon launch");
}

extern "C" int mnmt_debug_read(const void* d_x, size_t bytes, int reps, unsigned* d_sink, void* stream) {
  if (!d_x || !d_sink || bytes % 16 || reinterpret_cast<uintptr_t>(d_x) % 16 || reps < 1)
    return set_error(MNMT_E_INVALID_ARG,
                     "debug_read needs a 16-byte aligned buffer of a multiple of 16 bytes and reps >= 1");
  const hipError_t h = launch_debug_read(d_x, bytes, reps, d_sink, static_cast<hipStream_t>(stream));
  return h == hipSuccess ? MNMT_OK : hip_error(h, "debug_read launch");
}
