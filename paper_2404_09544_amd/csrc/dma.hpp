// LDS DMA helpers shared by the ring kernels (gemm.hip, train.hip).
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>

namespace gnnav {

// One wavefront-wide LDS DMA: lane l copies 16 bytes from its own global
// address g to LDS address lds + 16 * l (lds must be the same for every
// lane).  Issued from inline assembly, so the compiler does not know that
// LDS is written and adds no waits of its own: callers track completion
// with vmcnt (wait_vm) and publish it with a barrier.
__device__ __forceinline__ void dma16(const void *g, const void *lds) {
    const uint32_t la = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds);
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(la), "v"(g) : "memory", "m0");
}

// s_waitcnt vmcnt(N): at most N of this wavefront's vector loads pending.
template <int N>
__device__ __forceinline__ void wait_vm() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_s_waitcnt((15) | (7 << 4) | (0 << 8) | (3 << 14));   // lgkmcnt(0)
    asm volatile("s_barrier" ::: "memory");
}

}  // namespace gnnav
