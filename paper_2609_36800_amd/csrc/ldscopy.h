// Global -> LDS copies with explicitly managed completion (gfx950).
//
// global_load_lds_dwordx4 moves 16 bytes per lane from global memory straight
// into LDS (lane l's bytes land at the wave-uniform base + 16*l) without
// passing through VGPRs.  The copy is issued from inline asm so that the
// compiler does not model its LDS write: otherwise it waits for every copy in
// flight before each LDS read, which would collapse a multi-stage ring to one
// stage.  Completion is then established by hand: vector-memory loads retire
// in issue order, so s_waitcnt vmcnt(n) guarantees that all but the n most
// recently issued loads (copies included) have landed, and a barrier makes
// them visible to the other waves of the workgroup.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bitdelta {

typedef __attribute__((address_space(3))) void lds_void;

// s_waitcnt with vmcnt = N, lgkmcnt = 0, expcnt left alone (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vm_lgkm0() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4));
}

// Workgroup barrier without the implicit wait for all memory operations that
// __syncthreads() carries; the clobber keeps the compiler from moving memory
// accesses across it.
__device__ __forceinline__ void raw_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// One 16-byte-per-lane copy global -> LDS.  M0 holds the LDS base; the nop
// covers the M0-write -> LDS-DMA hazard.
__device__ __forceinline__ void copy16_to_lds(const void* src, void* lds_base) {
    const uint32_t lds_off = (uint32_t)(uintptr_t)(lds_void*)lds_base;
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
                 :: "s"(lds_off), "v"(src) : "memory", "m0");
}

// The same copy with the non-temporal hint, for cache lines read exactly once
// per launch (weight rows, and sign rows staged whole): measured 3-5% faster on
// the decode kernel's W stream than the default policy.  Lines that are read
// again keep the default: x (shared by every workgroup through L2) and sign
// rows fetched in pieces of a line over several tiles, which the hint turns
// into repeated HBM reads (up to 20% slower).
__device__ __forceinline__ void copy16_to_lds_nt(const void* src, void* lds_base) {
    const uint32_t lds_off = (uint32_t)(uintptr_t)(lds_void*)lds_base;
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off nt"
                 :: "s"(lds_off), "v"(src) : "memory", "m0");
}

// One 4-byte-per-lane copy global -> LDS: lane l's word lands at
// lds_base + 4*l (256 bytes per wave).
__device__ __forceinline__ void copy4_to_lds(const void* src, void* lds_base) {
    const uint32_t lds_off = (uint32_t)(uintptr_t)(lds_void*)lds_base;
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dword %1, off"
                 :: "s"(lds_off), "v"(src) : "memory", "m0");
}

}  // namespace bitdelta
