// KV-cache append / evict for gfx950.
//
// The K/V of the context chunks (c_0 and the previous chunks) are computed
// once and kept, so later chunks and both denoising steps never recompute
// them (TalkingMachines, Sec. 4.3, "KV & Embedding Cachings"). A new chunk's
// K and V arrive token-major, [B, n_tok, H, D]; the cache keeps them
// head-major, [B, H, capacity, D], so that the attention kernel streams each
// head's keys as one contiguous run. Writing a ring slot replaces, in place,
// the chunk that the window no longer needs: eviction moves no data.
//
// The copy is a pure HBM stream (read n_tok*H*D elements of K and of V, write
// as many): each thread moves 16-byte vectors, reads are contiguous in source
// order and every destination row of D elements is contiguous.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tm_internal.h"

namespace tmk {
namespace {

__global__ __launch_bounds__(256) void kv_append_kernel(const uint4* __restrict__ k_src,
                                                        const uint4* __restrict__ v_src,
                                                        uint4* __restrict__ k_pool,
                                                        uint4* __restrict__ v_pool, int64_t total,
                                                        int n_tok, int H, int vpr,
                                                        int64_t capacity, int64_t tok_offset) {
    // total = B * n_tok * H * vpr 16-byte vectors, enumerated in source order
    // (b, token, head, vector).
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < total;
         i += stride) {
        const int c = static_cast<int>(i % vpr);
        int64_t t = i / vpr;
        const int h = static_cast<int>(t % H);
        t /= H;
        const int tok = static_cast<int>(t % n_tok);
        const int64_t b = t / n_tok;
        const int64_t dst = ((b * H + h) * capacity + tok_offset + tok) * vpr + c;
        const uint4 kv = k_src[i];
        const uint4 vv = v_src[i];
        k_pool[dst] = kv;
        v_pool[dst] = vv;
    }
}

}  // namespace

hipError_t launch_kv_append(const void* k_src, const void* v_src, void* k_pool, void* v_pool,
                            int B, int n_tok, int H, int row_bytes, int64_t capacity,
                            int64_t tok_offset, hipStream_t s) {
    if (row_bytes % 16 != 0) return hipErrorInvalidValue;
    const int vpr = row_bytes / 16;
    const int64_t total = static_cast<int64_t>(B) * n_tok * H * vpr;
    if (total == 0) return hipSuccess;
    // Enough workgroups to cover the copy with a few vectors per thread while
    // keeping every CU busy.
    const int64_t want = (total + 256 * 4 - 1) / (256 * 4);
    const int blocks = static_cast<int>(want < 8192 ? (want < 1 ? 1 : want) : 8192);
    hipLaunchKernelGGL(kv_append_kernel, dim3(blocks), dim3(256), 0, s,
                       static_cast<const uint4*>(k_src), static_cast<const uint4*>(v_src),
                       static_cast<uint4*>(k_pool), static_cast<uint4*>(v_pool), total, n_tok, H,
                       vpr, capacity, tok_offset);
    return hipGetLastError();
}

}  // namespace tmk
