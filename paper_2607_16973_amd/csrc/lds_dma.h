// Direct global -> LDS loads and the waits and barriers around them (gfx950).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace tq {

// Loads of 16 bytes per lane straight into LDS: set_lds_base(b), then
// lds_dma16_at<K, NT>(src) puts lane l's 16 bytes from src at LDS byte
// address b + K KiB + 16 l (b wave-uniform).  The instruction offset moves
// both addresses, so it is taken off the source first.  Setting the base
// once per group of loads matters: a load must read M0 before it may change
// again.  The compiler does not see these loads: their completion is awaited
// with explicit vector-memory counter waits (wait_vmem) before the barrier
// that publishes the data (a wait on the counter also covers older accesses).
__device__ inline void set_lds_base(uint32_t lds_base) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0" :: "s"(__builtin_amdgcn_readfirstlane(lds_base))
                 : "memory");
}
// One such load with its own base (M0 set, then used).
__device__ inline void lds_dma16(const void *src, uint32_t lds_base) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
                 :: "s"(__builtin_amdgcn_readfirstlane(lds_base)), "v"(src) : "memory");
}
template <int K, bool NT>
__device__ inline void lds_dma16_at(const void *src) {
    const char *s = static_cast<const char *>(src) - K * 1024;
    if constexpr (NT)
        asm volatile("global_load_lds_dwordx4 %0, off offset:%1 nt" :: "v"(s), "i"(K * 1024) : "memory");
    else
        asm volatile("global_load_lds_dwordx4 %0, off offset:%1" :: "v"(s), "i"(K * 1024) : "memory");
}
// One load with a uniform source base and a 32-bit lane byte offset (the
// scalar-base form: no 64-bit address arithmetic per lane); lane l's 16
// bytes at sbase + voff go to LDS byte address lds_base + 16 l.
__device__ inline void lds_dma16_s(uint32_t voff, const void *sbase, uint32_t lds_base) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
                 :: "s"(__builtin_amdgcn_readfirstlane(lds_base)), "v"(voff), "s"(sbase)
                 : "memory");
}
// s_waitcnt until at most N vector-memory operations of this wave are
// outstanding (other counters unconstrained).
template <int N>
__device__ inline void wait_vmem() {
    static_assert(N >= 0 && N < 64, "vector-memory counter range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
// Barrier that orders LDS accesses only: outstanding global accesses of the
// wave (loads in flight, stores of an epilogue) need not complete here.
__device__ inline void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

}  // namespace tq
