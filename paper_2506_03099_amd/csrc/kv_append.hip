// KV-cache append / evict for gfx950.
//
// The K/V of the context chunks (c_0 and the previous chunks) are computed
// once and kept, so later chunks and both denoising steps never recompute
// them (TalkingMachines, Sec. 4.3, "KV & Embedding Cachings"). A new chunk's
// K and V arrive token-major, [B, n_tok, H, D]. The cache keeps K head-major,
// [B, H, capacity, D], so that the attention kernel streams each head's keys
// as one contiguous run, and V in blocks of 64 tokens stored dimension-major,
// [B, H, capacity / 64, D, 64], so that the attention kernel's V^T operand
// (8 consecutive keys of one dimension) is one 16-byte read. Writing a ring
// slot replaces, in place, the chunk that the window no longer needs:
// eviction moves no data.
//
// One workgroup per (batch, head, 64-token block of the cache touched by the
// chunk). K rows are copied with 16-byte vectors. V rows are staged in LDS
// and written back transposed, one 16-byte group of consecutive tokens of one
// dimension per store; the columns from n_tok up to the next multiple of 8
// are written as zeros, so that a 16-byte group the attention kernel reads
// never holds data of another region or unwritten memory.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tm_internal.h"

namespace tmk {
namespace {

constexpr int kAppendThreads = 256;

// EB: element bytes (2 or 4); D: head_dim.
template <int EB, int D>
__global__ __launch_bounds__(kAppendThreads) void kv_append_kernel(
    const unsigned char* __restrict__ k_src, const unsigned char* __restrict__ v_src,
    unsigned char* __restrict__ k_pool, unsigned char* __restrict__ v_pool, int n_tok, int H,
    int64_t capacity, int64_t tok_offset, int first_blk, int n_blk) {
    constexpr int B64 = kCacheBlock;
    constexpr int ROWB = D * EB;             // bytes of one token row of one head
    constexpr int VPR = ROWB / 16;           // 16-byte vectors per row
    constexpr int TPG = 16 / EB;             // tokens per 16-byte group of a V^T row
    constexpr int GPR = B64 / TPG;           // groups per V^T row
    constexpr int PITCH = ROWB / 4 + 1;      // LDS row pitch in 32-bit words (odd: no conflicts)
    static_assert(kCacheAlign % TPG == 0, "regions must start on whole 16-byte groups");
    __shared__ uint32_t tile[B64 * PITCH];

    const int bid = blockIdx.x;
    const int blk = first_blk + bid % n_blk;
    const int bh = bid / n_blk;
    const int h = bh % H;
    const int64_t b = bh / H;
    // Cache rows of this block that the append writes: [lo, hi), multiples of
    // kCacheAlign; rows at or past tok_offset + n_tok get zeros in V.
    const int64_t n_pad = (n_tok + kCacheAlign - 1) / kCacheAlign * kCacheAlign;
    const int64_t lo = max(static_cast<int64_t>(blk) * B64, tok_offset);
    const int64_t hi = min(static_cast<int64_t>(blk) * B64 + B64, tok_offset + n_pad);
    const int64_t src_stride = static_cast<int64_t>(H) * ROWB;  // bytes per source token
    const unsigned char* ks = k_src + b * n_tok * src_stride + static_cast<int64_t>(h) * ROWB;
    const unsigned char* vs = v_src + b * n_tok * src_stride + static_cast<int64_t>(h) * ROWB;
    const int64_t head = b * H + h;

    // K rows straight through; V rows into LDS (zeros past the chunk's end).
    for (int i = threadIdx.x; i < B64 * VPR; i += kAppendThreads) {
        const int r = i / VPR, c = i % VPR;
        const int64_t row = static_cast<int64_t>(blk) * B64 + r;
        if (row < lo || row >= hi) continue;
        const int64_t src = row - tok_offset;
        uint4 vv = make_uint4(0, 0, 0, 0);
        if (src < n_tok) {
            const uint4 kv = *reinterpret_cast<const uint4*>(ks + src * src_stride + c * 16);
            *reinterpret_cast<uint4*>(k_pool + (head * capacity + row) * ROWB + c * 16) = kv;
            vv = *reinterpret_cast<const uint4*>(vs + src * src_stride + c * 16);
        }
        uint32_t* t = &tile[r * PITCH + c * 4];
        t[0] = vv.x;
        t[1] = vv.y;
        t[2] = vv.z;
        t[3] = vv.w;
    }
    __syncthreads();

    // V^T: row d of the block holds the 64 tokens' element d; each thread
    // writes one 16-byte group (TPG consecutive tokens) of one row.
    unsigned char* vblk = v_pool + ((head * (capacity / B64)) + blk) * static_cast<int64_t>(D) * B64 * EB;
    for (int i = threadIdx.x; i < D * GPR; i += kAppendThreads) {
        const int d = i / GPR, g = i % GPR;
        const int64_t row0 = static_cast<int64_t>(blk) * B64 + g * TPG;
        if (row0 < lo || row0 >= hi) continue;
        uint32_t w[4];
        if constexpr (EB == 4) {
#pragma unroll
            for (int e = 0; e < 4; ++e) w[e] = tile[(g * TPG + e) * PITCH + d];
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int r0 = g * TPG + 2 * e;
                const uint32_t a0 = tile[r0 * PITCH + d / 2] >> (16 * (d & 1));
                const uint32_t a1 = tile[(r0 + 1) * PITCH + d / 2] >> (16 * (d & 1));
                w[e] = (a0 & 0xFFFFu) | (a1 << 16);
            }
        }
        *reinterpret_cast<uint4*>(vblk + (static_cast<int64_t>(d) * B64 + g * TPG) * EB) =
            make_uint4(w[0], w[1], w[2], w[3]);
    }
}

template <int EB, int D>
hipError_t launch(const void* k_src, const void* v_src, void* k_pool, void* v_pool, int B,
                  int n_tok, int H, int64_t capacity, int64_t tok_offset, hipStream_t s) {
    const int64_t n_pad = (n_tok + kCacheAlign - 1) / kCacheAlign * kCacheAlign;
    const int64_t first = tok_offset / kCacheBlock;
    const int64_t last = (tok_offset + n_pad - 1) / kCacheBlock;
    const int64_t n_blk = last - first + 1;
    const int64_t grid = n_blk * B * H;
    if (grid > INT32_MAX) return hipErrorInvalidValue;
    hipLaunchKernelGGL((kv_append_kernel<EB, D>), dim3(static_cast<unsigned>(grid)),
                       dim3(kAppendThreads), 0, s, static_cast<const unsigned char*>(k_src),
                       static_cast<const unsigned char*>(v_src), static_cast<unsigned char*>(k_pool),
                       static_cast<unsigned char*>(v_pool), n_tok, H, capacity, tok_offset,
                       static_cast<int>(first), static_cast<int>(n_blk));
    return hipGetLastError();
}

}  // namespace

hipError_t launch_kv_append(const void* k_src, const void* v_src, void* k_pool, void* v_pool,
                            int B, int n_tok, int H, int D, int elem_bytes, int64_t capacity,
                            int64_t tok_offset, hipStream_t s) {
    const int64_t n_pad = (static_cast<int64_t>(n_tok) + kCacheAlign - 1) / kCacheAlign * kCacheAlign;
    if (n_tok < 1 || tok_offset % kCacheAlign != 0 || capacity % kCacheBlock != 0 ||
        tok_offset + n_pad > capacity)
        return hipErrorInvalidValue;
    if (elem_bytes == 2 && D == 128)
        return launch<2, 128>(k_src, v_src, k_pool, v_pool, B, n_tok, H, capacity, tok_offset, s);
    if (elem_bytes == 2 && D == 64)
        return launch<2, 64>(k_src, v_src, k_pool, v_pool, B, n_tok, H, capacity, tok_offset, s);
    if (elem_bytes == 4 && D == 128)
        return launch<4, 128>(k_src, v_src, k_pool, v_pool, B, n_tok, H, capacity, tok_offset, s);
    if (elem_bytes == 4 && D == 64)
        return launch<4, 64>(k_src, v_src, k_pool, v_pool, B, n_tok, H, capacity, tok_offset, s);
    return hipErrorInvalidValue;
}

}  // namespace tmk
