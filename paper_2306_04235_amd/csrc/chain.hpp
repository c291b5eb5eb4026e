// chain.hpp -- the hand-off between consecutive kernels of a translation
// that run on two alternating streams (StepChain in internal.h): a kernel
// issues the loads that do not depend on its predecessor, waits on the
// predecessor's per-block flag words, and stores its own when done.
#pragma once

#include "internal.h"

namespace mnmt {

// Waits for the previous kernel of a translation's chain (see StepChain):
// thread i polls the flag word of block i (relaxed, agent scope), then each
// polling wave takes an acquire fence and the block a barrier, after which
// every thread sees the previous kernel's writes.  Called after the weight loads
// are issued, so they arrive while the previous kernel still runs.
__device__ __forceinline__ void chain_wait(const StepChain& c) {
  if (!c.wait) return;
  const int tid = threadIdx.x;
  if (tid < c.nwait) {
    const unsigned* w = c.wait + (blockIdx.x % chain_copies(c.nwait)) * kChainCopyStride + tid;
    unsigned n = 0;
    while (__hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < c.want) {
      __builtin_amdgcn_s_sleep(2);
      if (++n >= kChainSpinLimit) {  // never in a correct chain: record it and go on
        __hip_atomic_fetch_or(c.err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
    }
  }
  // the acquire (an invalidation of the CU's caches) once per polling wave;
  // the barrier then orders every wave's loads after it
  if ((int)(tid & ~63) < c.nwait) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  __syncthreads();
}

// A global store that a later kernel of the chain reads: a relaxed
// agent-scope atomic store, which goes through to the device's point of
// coherence instead of staying in the writer's L2 (each XCD has its own).
// With every such write made this way (and the accumulators' agent-scope
// atomics), chain_signal only waits for the writes to complete and needs no
// write-back of the L2, which an agent-scope release performs.
template <class T>
__device__ __forceinline__ void chain_store(T* p, T v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The flag word of block `bid` of a kernel role of `nblk` blocks (in every
// copy), stored once every wave's writes (chain_store, atomics) have
// completed.
__device__ __forceinline__ void chain_signal_as(const StepChain& c, int bid, int nblk) {
  if (!c.done) return;
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0);  // this wave's stores and atomics complete
  __syncthreads();                // ... and every other wave's
  if ((int)threadIdx.x < chain_copies(nblk))
    __hip_atomic_store(c.done + threadIdx.x * kChainCopyStride + bid, c.val, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void chain_signal(const StepChain& c) {
  chain_signal_as(c, blockIdx.x, gridDim.x);
}

}  // namespace mnmt
