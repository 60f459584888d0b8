// Synchronisation helpers for kernels that stage operands through LDS with
// direct-to-LDS loads (global_load_lds).
#pragma once
#include <hip/hip_runtime.h>

namespace gvc {

// Workgroup barrier for pipelines fed by direct-to-LDS loads.
// __syncthreads() also fences memory, and that fence makes every wave wait
// for all of its outstanding global loads (vmcnt 0), prefetches of later
// steps included, before the barrier.  Here the caller first waits (with
// s_waitcnt) for exactly the loads the next step reads; the empty asm
// statements keep the compiler from moving memory accesses across the
// barrier.  Only for LDS data written by those loads or read before the
// previous barrier.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Waits until at most N of this wave's vector memory loads are outstanding
// (direct-to-LDS loads included; they complete in issue order).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}

}  // namespace gvc
