// noalloc.hip -- the fused logits + arg-max over a fragment-order weight
// (MNMT_EPI_ARGMAX_PARTIAL_PACKED of mnmt_qlinear) for callers that cannot
// allocate device memory: the per-block partial keys live in a file-scope
// device array instead of a caller buffer, and a second kernel reduces them
// to each row's arg-max key and index.
#include <mutex>
#include <vector>

#include "canon.hpp"
#include "internal.h"

namespace mnmt {
namespace {

constexpr int kNoAllocRows = 2;             // rows of the batch-1 logits kernel
constexpr int kNoAllocMaxN = 262144;        // outputs (vocabulary rows)
constexpr int kNoAllocMaxPartials = 2048;   // step_logits_blocks(kNoAllocMaxN): 128 outputs per block
constexpr size_t kScratchWords = (size_t)kNoAllocRows * kNoAllocMaxPartials;  // 32 KiB

// Each GPU the library runs on holds its own copy until the process ends.
// Host code never uses this name as an address: it takes the device address
// from hipGetSymbolAddress (per device, see scratch_ptr).
__device__ __align__(256) unsigned long long scratch[kScratchWords];

std::mutex g_mu;
std::vector<unsigned long long*> g_ptr;  // device address of `scratch`, by device id

// The current device's address of `scratch`, looked up on the first call on
// that device (with it current) and kept.
int scratch_ptr(unsigned long long** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_error(e, "hipGetDevice");
  std::lock_guard<std::mutex> lock(g_mu);
  if ((int)g_ptr.size() <= dev) g_ptr.resize(dev + 1, nullptr);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_error(e, "hipGetSymbolAddress(scratch)");
    if (!p) return set_error(MNMT_E_HIP, "hipGetSymbolAddress(scratch) returned null");
    g_ptr[dev] = static_cast<unsigned long long*>(p);
  }
  *out = g_ptr[dev];
  return MNMT_OK;
}

// One block per row: the largest of the row's P partial keys (value key << 32
// | ~index, so the maximum is the arg max with the smallest index among equal
// maxima), stored with its index.
__global__ __launch_bounds__(256) void k_reduce_partials(const unsigned long long* __restrict__ part, int P,
                                                         unsigned long long* key_out, int32_t* tok_out) {
  const int m = blockIdx.x;
  unsigned long long b = 0ull;
  for (int i = threadIdx.x; i < P; i += blockDim.x) {
    const unsigned long long v = part[(size_t)m * P + i];
    b = v > b ? v : b;
  }
  b = wave_max_u64(b);
  __shared__ unsigned long long wbest[4];
  if ((threadIdx.x & 63) == 0) wbest[threadIdx.x >> 6] = b;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < 4; ++w) b = wbest[w] > b ? wbest[w] : b;
    if (key_out) key_out[m] = b;
    if (tok_out) tok_out[m] = unpack_index(b);
  }
}

}  // namespace
}  // namespace mnmt

using namespace mnmt;

extern "C" int mnmt_logits_argmax_noalloc(const int8_t* d_X, const int8_t* d_Wp, const float* d_scale, int M, int K,
                                          int N, unsigned long long* d_key, int32_t* d_tok, void* stream) {
  if (M < 1 || M > kNoAllocRows || K < 64 || K % 64 || K > 512 || N < 1 || N > kNoAllocMaxN)
    return set_error(MNMT_E_INVALID_ARG,
                     "logits_argmax_noalloc takes 1 <= M <= 2, K a multiple of 64 up to 512 and 1 <= N <= 262144 "
                     "(its static scratch holds 2 x 2048 partial keys)");
  if (!step_logits_fits(M, K) || step_logits_blocks(N) > kNoAllocMaxPartials)
    return set_error(MNMT_E_INVALID_ARG, "shape exceeds the static scratch");
  if (!d_X || !d_Wp || !d_scale || (!d_key && !d_tok)) return set_error(MNMT_E_INVALID_ARG, "null device pointer");
  if (reinterpret_cast<uintptr_t>(d_X) % 16 || reinterpret_cast<uintptr_t>(d_Wp) % 16)
    return set_error(MNMT_E_INVALID_ARG, "X and W must be 16-byte aligned");
  unsigned long long* part = nullptr;
  int rc = scratch_ptr(&part);
  if (rc) return rc;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  // the same kernel as MNMT_EPI_ARGMAX_PARTIAL_PACKED: every block stores its
  // partial key of every row (plain stores, so nothing needs clearing)
  StepLogits g{};
  g.R = M;
  g.d = K;
  g.V = N;
  g.E = d_Wp;
  g.frag = true;
  g.c_out = d_scale;
  g.slots = part;
  g.nslots = step_logits_blocks(N);
  g.x_i8 = d_X;
  hipError_t h = launch_step_logits(StepIn{}, g, s);
  if (h != hipSuccess) return hip_error(h, "logits launch");
  hipLaunchKernelGGL(k_reduce_partials, dim3(M), dim3(256), 0, s, part, g.nslots, d_key, d_tok);
  h = hipGetLastError();
  return h == hipSuccess ? MNMT_OK : hip_error(h, "partial reduction launch");
}
