// Global-to-LDS loads that bypass registers (global_load_lds_dword /
// global_load_lds_dwordx4) and the explicit waits and barrier that go with
// them; shared by the matrix-core scans.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sense {

// Waits until at most N vector-memory operations of this wave are still
// outstanding (they complete in issue order).  Also a compiler barrier for
// memory accesses.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// 16 (or 4) bytes per lane from global memory straight into LDS: lane l's
// bytes land at lds + 16*l (4*l); lds is wave-uniform.  Written as inline
// assembly so that the compiler's wait-count model does not see an LDS write
// it cannot attribute to a ring slot (it would then wait for every
// outstanding load before each LDS read); the waits are explicit instead.
// m0 is a reserved register: the compiler never keeps a value in it across
// code it does not control and sets it right before each of its own uses, so
// listing it as clobbered here is safe (clang warns about it regardless).
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(const void* g, void* lds) {
    const uint32_t base = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds);
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(base)
                 : "memory", "m0");
}
// The same with the non-temporal hint, for the key stream: every key byte is
// used once per scan, and without the hint the stream evicts the query
// fragments, which every block re-reads, from L2 (at 64 queries with the
// hi/lo split those are 2 MiB per XCD; measured: 16 % more HBM traffic than
// the keys alone).
__device__ __forceinline__ void dma16_nt(const void* g, void* lds) {
    const uint32_t base = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds);
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off nt" ::"v"(g), "s"(base)
                 : "memory", "m0");
}
__device__ __forceinline__ void dma4(const void* g, void* lds) {
    const uint32_t base = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds);
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dword %0, off" ::"v"(g), "s"(base)
                 : "memory", "m0");
}
#pragma clang diagnostic pop

// Workgroup barrier without the memory fence __syncthreads() adds (the fence
// would wait for every outstanding load, draining the pipeline).  LDS data
// written by DMA is complete once the issuing wave's vmcnt wait returns.
__device__ __forceinline__ void barrier_no_fence() { asm volatile("s_barrier" ::: "memory"); }

}  // namespace sense
