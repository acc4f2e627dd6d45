// Workgroup barrier for data exchanged through LDS only.
#pragma once

#include <hip/hip_runtime.h>

namespace aqlm {

// Orders and completes this wave's LDS accesses (and nothing else) before the
// barrier.  Global loads issued earlier stay in flight across it, whereas the
// fence of __syncthreads also waits for them (loads and stores share one
// counter), which would expose the latency of every prefetch issued before
// the barrier.  Only for barriers whose data dependences go through LDS.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

}  // namespace aqlm
