// Direct global->LDS staging and wait helpers shared by the lm-head kernels
// (gfx950: 64 LDS banks of 4 bytes, global_load_lds_dwordx4).
#pragma once

#include "device_common.h"
#include "tile_index.h"

namespace rlk {

// 16 bytes global -> LDS, bypassing the registers.  Lane i of a wave writes
// LDS bytes [base + 16 i, +16) (base in M0, wave-uniform), so one instruction
// fills 1 KB contiguously.  Issued as inline assembly: the compiler then does
// not know that it writes LDS and does not put a wait for all loads in flight
// in front of every LDS read (it cannot tell the stage buffers apart); the
// kernels order these loads against their LDS reads with explicit waits.
// M0 is an input operand ("{m0}"), so the compiler itself writes it and knows
// that it holds the LDS base; the asm only reads it.  The leading s_nop is
// the one wait state the ISA requires between an SALU write of M0 and an LDS
// DMA instruction that reads it (the compiler's hazard tracking does not look
// inside the asm).
//
// LDS destinations are passed as 32-bit LDS byte addresses: the address of a
// __shared__ array is taken once (lds_addr) and each load adds a wave-uniform
// offset on the scalar unit.  Converting a generic pointer at every load
// would cost a 64-bit add, a null check and a select per load.
__device__ __forceinline__ uint32_t lds_addr(const void *l) {
    typedef __attribute__((address_space(3))) const unsigned char lds_u8;
    return __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_u8 *)(l))));
}

// A value the same in every lane of the wave, read first-lane so the compiler
// keeps it (and what is computed from it) in SGPRs.  The tile coordinates come
// out of 64-bit divisions the compiler expands on the VALU.  The builtin
// returns a signed int: each half goes through uint32_t before widening, or
// a low half with bit 31 set would sign-extend into the high half.
__device__ __forceinline__ int64_t uniform64(int64_t x) {
    const uint64_t u = static_cast<uint64_t>(x);
    const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(static_cast<uint32_t>(u))));
    const uint32_t hi =
        static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(static_cast<uint32_t>(u >> 32))));
    return static_cast<int64_t>((static_cast<uint64_t>(hi) << 32) | lo);
}

// A wave-uniform global base in SGPRs plus a per-lane 32-bit byte offset
// (the global_load_lds "saddr" form): no 64-bit address arithmetic per lane.
// The base must be computed on the scalar unit: the compiler's hazard
// tracking does not see that the asm's VMEM instruction reads those SGPRs, so
// a VALU write of them (a v_readfirstlane) right before it would need 5 wait
// states it does not get.  build.py checks the gfx950 assembly for that.
// `lds` is the destination's LDS byte address (lds_addr + offset).
__device__ __forceinline__ void load_lds16_s(const void *base, uint32_t voff, uint32_t lds) {
    asm volatile(
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %0, %1"
        :
        : "v"(voff), "s"(base), "{m0}"(lds)
        : "memory");
}

// Wait until at most N vector-memory operations of this wave are outstanding.
// The global->LDS loads are tracked by this counter; the compiler does not see
// when their LDS bytes are read, so the waits are explicit.
template <int N>
__device__ __forceinline__ void wait_vm() { asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory"); }

__device__ __forceinline__ void wait_lds() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

__device__ __forceinline__ void barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

}  // namespace rlk
