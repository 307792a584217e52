// Direct-to-LDS staging helpers shared by the kernels that stream tiles through LDS
// (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace moe {

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt field is 6 bits");
    // gfx9 s_waitcnt: vmcnt[3:0] | expcnt[6:4]=7 | lgkmcnt[11:8]=15 | vmcnt[5:4] at [15:14]
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt((15) | (7 << 4) | (0 << 8) | (3 << 14)); }

// Wait until at most `newer` stages of LPW loads each are still in flight.
template <int LPW, int NS>
__device__ __forceinline__ void wait_stages(int newer) {
    static_assert(NS >= 2 && NS <= 6, "pipeline depth");
    if (NS > 5 && newer >= 4) { wait_vmcnt<(NS > 5 ? 4 * LPW : 0)>(); return; }
    if (NS > 4 && newer >= 3) { wait_vmcnt<(NS > 4 ? 3 * LPW : 0)>(); return; }
    if (NS > 3 && newer >= 2) { wait_vmcnt<(NS > 3 ? 2 * LPW : 0)>(); return; }
    if (NS > 2 && newer >= 1) { wait_vmcnt<(NS > 2 ? LPW : 0)>(); return; }
    wait_vmcnt<0>();
}

// A wave-uniform value in scalar registers (the asm operands below must be scalar even where
// the compiler cannot prove uniformity itself).
__device__ __forceinline__ const unsigned char* uniform_ptr(const void* p) {
    const uint64_t v = reinterpret_cast<uintptr_t>(p);
    const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v));
    const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v >> 32));
    return reinterpret_cast<const unsigned char*>((static_cast<uint64_t>(hi) << 32) | lo);
}

// 16 bytes per lane from global memory straight into LDS: lane l's bytes come from
// base + voff(l) and land at lds + 16 l (the LDS address is wave-uniform and goes through
// M0; base is a wave-uniform 64-bit address in scalar registers, voff a 32-bit per-lane
// byte offset).  Issued as inline assembly on purpose: the compiler tracks the builtin
// form as an LDS write and then waits for it (vmcnt(0)) before every later LDS read it
// cannot prove disjoint -- which would make the prefetched stages synchronous.  The kernels
// order these loads themselves (vmcnt waits before the stage barrier, and a stage buffer
// is refilled only after the barrier that follows every wave's reads of it).  The "memory"
// clobber keeps the compiler from moving LDS accesses across the issue.
__device__ __forceinline__ void load_lds16(const unsigned char* base, uint32_t voff, uint32_t lds_addr) {
    base = uniform_ptr(base);
    lds_addr = __builtin_amdgcn_readfirstlane(lds_addr);
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2" ::"s"(lds_addr), "v"(voff), "s"(base)
                 : "memory", "m0");
}

// LDS byte address of a shared-memory pointer (wave-uniform).
__device__ __forceinline__ uint32_t lds_address(const void* p) {
    return __builtin_amdgcn_readfirstlane(
        static_cast<uint32_t>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) const void*)p)));
}

// Ask the scheduler to spread a step's LDS fragment reads between its MFMAs (one read after
// every M / R MFMAs) instead of issuing them as one burst: a burst holds up the next MFMA
// issue, and with one or two waves per SIMD nothing else fills the matrix core meanwhile.
template <int M, int R>
__device__ __forceinline__ void interleave_reads() {
    constexpr int per = M / R > 0 ? M / R : 1;
#pragma unroll
    for (int k = 0; k < R; ++k) {
        __builtin_amdgcn_sched_group_barrier(0x008, per, 0);  // MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);    // LDS read
    }
    __builtin_amdgcn_sched_group_barrier(0x008, M - per * R > 0 ? M - per * R : 0, 0);
}

// Bare workgroup barrier.  A fenced barrier (__syncthreads, or even an LDS-only fence)
// makes the compiler wait for every direct-to-LDS load in flight, which would drain the
// prefetched stages this pipeline keeps in flight across the barrier.  The empty asm
// statements with a memory clobber keep the compiler from moving LDS reads across it.
__device__ __forceinline__ void stage_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

}  // namespace moe
