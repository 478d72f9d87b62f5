// Device-side helpers shared by the attention kernels (attn_fwd.hip,
// audio_attn.hip, attn_bwd.hip). Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tmk {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr float kNegInf = -__builtin_inff();

// Workgroups are dispatched round-robin over the 8 XCDs (each with its own L2).
// Renumber them so that consecutive logical ids (workgroups that read the
// same K/V) land on the same XCD.
__device__ __forceinline__ int xcd_logical_id(int bid, int total) {
    constexpr int kXcds = 8;
    const int per = total / kXcds, rem = total % kXcds;
    const int x = bid % kXcds, j = bid / kXcds;
    return x * per + min(x, rem) + j;
}

// Row of a 32-key block that lane l32 feeds to the score MFMA
// S^T = K Q^T (v_mfma_f32_32x32x16_bf16) so that P can feed the P V MFMA
// from registers: bits 2 and 3 of the row swapped. The S^T output register i
// of a lane in half-wave hw then holds key 16*(i/8) + 8*hw + i%8 of the
// block, so the 8 P^T elements a lane feeds to a 16-key MFMA step are 8
// consecutive keys.
__device__ __forceinline__ int k_perm(int r) { return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1); }

// Position of 16-byte chunk c of row `row` in a K or row-major V tile of D
// bf16 per row in LDS: c ^ lds_swizzle<D>(row). Low three bits: a
// permutation of 0..7 over any 8 aligned rows (K reads of one chunk from 8
// consecutive rows hit 8 distinct 16-byte bank groups), with bits 1-2
// distinct over any 4 aligned rows (the transposing V reads' chunk pairs
// {p, p^1} of 4 consecutive rows are disjoint). Bit 3 (rows of 16 chunks
// only) separates rows r and r + 8. Depends on row % 16 only.
template <int D>
__device__ __forceinline__ int lds_swizzle(int row) {
    const int low = 2 * (row & 3) + ((row >> 2) & 1);
    return D == 128 ? low + 8 * ((row >> 3) & 1) : low;
}

// Position of 16-byte chunk c of row `row` in an LDS tile of D bf16 per row
// read both by rows and by transposing reads: c ^ tr_swizzle<D>(row). LDS
// serves 64 banks of 4 bytes: a 16-byte read per lane covers 16 lanes per
// cycle (16 consecutive rows of one chunk: distinct chunk slots), an 8-byte
// transposing read 32 lanes (4 consecutive rows, 4 chunks each: distinct
// 64-byte slot groups). D = 128: a permutation of 0..15 over 16 rows whose
// bits 2-3 differ over 4 aligned rows; D = 64 (two rows per 256 bytes): the
// same within the even and within the odd rows.
template <int D>
__device__ __forceinline__ int tr_swizzle(int row) {
    return D == 128 ? 4 * (row & 3) + ((row >> 2) & 3) : 4 * ((row >> 1) & 1) + ((row >> 2) & 3);
}

// s_waitcnt immediate (gfx9 encoding) for vmcnt(0), expcnt and lgkmcnt unconstrained.
constexpr int kWaitVmcnt0 = 0x0F70;
// s_waitcnt immediate for lgkmcnt(0), vmcnt and expcnt unconstrained.
constexpr int kWaitLgkmcnt0 = 0xC07F;

// A pointer that is the same in every lane, held in scalar registers.
__device__ __forceinline__ const void* uniform_ptr(const void* p) {
    const uint64_t v = reinterpret_cast<uint64_t>(p);
    const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v));
    const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v >> 32));
    return reinterpret_cast<const void*>((static_cast<uint64_t>(hi) << 32) | lo);
}

// Two direct global->LDS loads (global_load_lds_dwordx4) of 16 bytes per lane:
// load n reads from the wave-uniform base sbase<n> plus the lane's byte offset
// voff<n>, and lane l's bytes land at LDS address lds<n> + 16 * l. The LDS
// address goes through M0 (saved and restored); an SALU write of M0 needs one
// wait state before an LDS-DMA instruction (or anything else) reads it, hence
// the s_nop after each write. Written as inline assembly so that these loads
// stay out of the compiler's wait bookkeeping, which would otherwise make LDS
// reads of one tile wait for the loads of later tiles; the kernel waits for
// them explicitly before the barrier that publishes a tile.
__device__ __forceinline__ void lds_dma16x2(const void* sbase0, uint32_t voff0, uint32_t lds0,
                                            const void* sbase1, uint32_t voff1, uint32_t lds1) {
    uint32_t saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %1\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %2, %3\n\t"
        "s_mov_b32 m0, %4\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %5, %6\n\t"
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0"
        : "=&s"(saved)
        : "s"(lds0), "v"(voff0), "s"(sbase0), "s"(lds1), "v"(voff1), "s"(sbase1));
}

// One direct global->LDS load (global_load_lds_dword) of 4 bytes per lane into
// lds + 4 * l for each of two sources, as lds_dma16x2 otherwise.
__device__ __forceinline__ void lds_dma4x2(const void* sbase0, uint32_t voff0, uint32_t lds0,
                                           const void* sbase1, uint32_t voff1, uint32_t lds1) {
    uint32_t saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %1\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dword %2, %3\n\t"
        "s_mov_b32 m0, %4\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dword %5, %6\n\t"
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0"
        : "=&s"(saved)
        : "s"(lds0), "v"(voff0), "s"(sbase0), "s"(lds1), "v"(voff1), "s"(sbase1));
}

// One direct global->LDS load (global_load_lds_dwordx4) of 16 bytes per lane
// into lds + 16 * l, as lds_dma16x2 otherwise.
__device__ __forceinline__ void lds_dma16(const void* sbase, uint32_t voff, uint32_t lds) {
    uint32_t saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %1\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %2, %3\n\t"
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0"
        : "=&s"(saved)
        : "s"(lds), "v"(voff), "s"(sbase));
}

// 16-byte store at system scope (sc0 sc1), written through the L2. A plain
// store leaves its line dirty in the L2, and the dirty lines are written back
// when the kernel ends, after its last wave: for a kernel whose output is
// mostly stores (tens of MB) that is a serial tail of a few
// microseconds, where written-through lines drain while the kernel runs. The
// s_nop covers the store reading its data registers after issue.
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void store16_through(void* p, u32x4_t v) {
    asm volatile("global_store_dwordx4 %0, %1, off sc0 sc1\n\ts_nop 1" ::"v"(p), "v"(v) : "memory");
}

// Wait until every direct global->LDS load issued by this wave has written
// LDS. The barrier that publishes a tile only orders LDS operations; the
// direct loads count as vector-memory operations, so each wave waits for its
// own before the barrier, and after the barrier the whole tile is in place.
__device__ __forceinline__ void wait_lds_dma() { __builtin_amdgcn_s_waitcnt(kWaitVmcnt0); }

}  // namespace tmk
