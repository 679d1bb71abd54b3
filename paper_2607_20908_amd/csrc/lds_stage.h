// Direct global->LDS staging and wait helpers shared by the lm-head kernels
// (gfx950: 64 LDS banks of 4 bytes, global_load_lds_dwordx4).
#pragma once

#include "device_common.h"

namespace rlk {

// 16 bytes global -> LDS, bypassing the registers.  Lane i of a wave writes
// LDS bytes [base + 16 i, +16) (base in M0, wave-uniform), so one instruction
// fills 1 KB contiguously.  Issued as inline assembly: the compiler then does
// not know that it writes LDS and does not put a wait for all loads in flight
// in front of every LDS read (it cannot tell the stage buffers apart); the
// kernels order these loads against their LDS reads with explicit waits.
__device__ __forceinline__ void load_lds16(const uint16_t *g, uint16_t *l) {
    typedef __attribute__((address_space(3))) uint16_t lds_u16;
    const uint32_t lds_addr = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_u16 *)(l)));
    asm volatile(
        "s_mov_b32 m0, %1\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %0, off"
        :
        : "v"(g), "s"(__builtin_amdgcn_readfirstlane(lds_addr))
        : "memory", "m0");
}

// The same with a wave-uniform base in SGPRs and a per-lane 32-bit byte offset
// (the global_load_lds "saddr" form): no 64-bit address arithmetic per lane.
__device__ __forceinline__ void load_lds16_s(const void *base, uint32_t voff, uint16_t *l) {
    typedef __attribute__((address_space(3))) uint16_t lds_u16;
    const uint32_t lds_addr = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_u16 *)(l)));
    asm volatile(
        "s_mov_b32 m0, %2\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %0, %1"
        :
        : "v"(voff), "s"(base), "s"(__builtin_amdgcn_readfirstlane(lds_addr))
        : "memory", "m0");
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

// Element offset of 16-byte chunk c (0..7) of row `row` in a [rows][64] bf16
// stage image.  Rows are 128 bytes, so two rows share one 256-byte window of
// the 64 LDS banks; XOR-ing the chunk with row bits 1..3 gives the 16 rows
// that one ds_read_b128 pass serves (same chunk, consecutive rows) 16 distinct
// 16-byte slots of that window.
__device__ __forceinline__ int op_off(int row, int c) { return row * 64 + ((c ^ ((row >> 1) & 7)) << 3); }

// Logical tile index -> (n-tile, m-tile): groups of 4 m-tiles sweep the
// n-tiles together, so an n-tile's operand is fetched into an L2 once for 4
// m-tiles while the m-tiles' operand stays resident in L2 / the MALL.
__device__ __forceinline__ void tile_of_logical(int64_t L, int64_t nnt, int64_t nmt, int64_t *nt, int64_t *mt) {
    constexpr int64_t GR = 4;
    const int64_t group = L / (GR * nnt);
    const int64_t in = L % (GR * nnt);
    const int64_t rows_in_group = min(GR, nmt - group * GR);
    *mt = group * GR + in % rows_in_group;
    *nt = in / rows_in_group;
}

// Launch index -> (n-tile, m-tile) for a launch over logical tiles [base,
// base + count).  The hardware hands consecutive workgroups to the 8 XCDs in
// turn; renumbering gives each XCD a contiguous run of logical tiles, so the
// sharing above happens inside one XCD's L2.
__device__ __forceinline__ void tile_of(int64_t b, int64_t count, int64_t base, int64_t nnt, int64_t nmt,
                                        int64_t *nt, int64_t *mt) {
    const int64_t full = count / 8 * 8;
    const int64_t L = b < full ? (b % 8) * (count / 8) + b / 8 : b;
    tile_of_logical(base + L, nnt, nmt, nt, mt);
}

}  // namespace rlk
