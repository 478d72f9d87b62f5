// Device-side helpers shared by the attention kernels (attn_fwd.hip,
// audio_attn.hip). Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>

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

}  // namespace tmk
