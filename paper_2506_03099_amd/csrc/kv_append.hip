// KV-cache append / evict, and the fused K/V producer, for gfx950.
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
//
// The fused producer is the same kernel with the chunk's queries and keys
// RMS-normalised on the way (the student keeps the query/key normalisation of
// its WAN2.1 teacher, Sec. 4.1, and the cached keys are the normalised ones):
// the lanes holding one (token, head) row reduce its sum of squares with DPP
// moves, scale by 1/sqrt(mean + eps) and the per-(head, dim) gain in fp32,
// and store the rounded result (queries to q_out, keys to the cache). One pass
// over q, k and v instead of a normalisation pass plus the append.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tm_device.h"
#include "tm_internal.h"

namespace tmk {
namespace {

constexpr int kAppendThreads = 256;

// Elements of one 16-byte vector as fp32, and back (RNE for bf16).
template <int EB>
__device__ __forceinline__ void unpack16(const uint4& u, float (&x)[16 / EB]) {
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
    if constexpr (EB == 4) {
#pragma unroll
        for (int e = 0; e < 4; ++e) x[e] = __uint_as_float(w[e]);
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            x[2 * e] = __uint_as_float(w[e] << 16);
            x[2 * e + 1] = __uint_as_float(w[e] & 0xFFFF0000u);
        }
    }
}
template <int EB>
__device__ __forceinline__ uint4 pack16(const float (&x)[16 / EB]) {
    uint32_t w[4];
    if constexpr (EB == 4) {
#pragma unroll
        for (int e = 0; e < 4; ++e) w[e] = __float_as_uint(x[e]);
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const __bf16 lo = static_cast<__bf16>(x[2 * e]), hi = static_cast<__bf16>(x[2 * e + 1]);
            w[e] = static_cast<uint32_t>(__builtin_bit_cast(uint16_t, lo)) |
                   (static_cast<uint32_t>(__builtin_bit_cast(uint16_t, hi)) << 16);
        }
    }
    return make_uint4(w[0], w[1], w[2], w[3]);
}

// Sum over the VPR consecutive lanes that hold one row, left in every one of
// them: DPP swaps inside quads, then the half-row mirror (8 lanes) or two
// rotations inside the 16-lane row, then lane^16 for 32-lane rows.
template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
template <int VPR>
__device__ __forceinline__ float row_sum(float s) {
    static_assert(VPR == 8 || VPR == 16 || VPR == 32, "8, 16 or 32 lanes per row");
    s += dpp_f<0xB1>(s);  // quad_perm [1, 0, 3, 2]
    s += dpp_f<0x4E>(s);  // quad_perm [2, 3, 0, 1]
    if constexpr (VPR == 8) {
        s += dpp_f<0x141>(s);  // row_half_mirror: the other quad of the 8
    } else {
        s += dpp_f<0x124>(s);  // row_ror:4
        s += dpp_f<0x128>(s);  // row_ror:8
        if constexpr (VPR == 32) s += __shfl_xor(s, 16);
    }
    return s;
}

// RMS normalisation of one (token, head) row held by VPR consecutive lanes,
// 16 bytes each: x <- x / sqrt(mean(x^2) + eps) * gain (g: this lane's gain
// elements; ones without a gain, which leaves the product exact). Every lane
// of the wave takes part in the reduction (rows outside the block carry zeros).
template <int EB, int D, int VPR>
__device__ __forceinline__ void rms_normalise_row(float (&x)[16 / EB], const float (&g)[16 / EB],
                                                  float eps) {
    constexpr int N = 16 / EB;
    float ss = 0.f;
#pragma unroll
    for (int e = 0; e < N; ++e) ss = fmaf(x[e], x[e], ss);
    ss = row_sum<VPR>(ss);
    const float r = 1.f / sqrtf(ss / static_cast<float>(D) + eps);
#pragma unroll
    for (int e = 0; e < N; ++e) x[e] = x[e] * r * g[e];
}

// This lane's N gain elements of a (head, dim) row (16-byte aligned: the
// host checks 16-byte alignment of the gain arrays), or ones.
template <int N>
__device__ __forceinline__ void load_gain(const float* gain, int c, float (&g)[N]) {
    if (gain == nullptr) {
#pragma unroll
        for (int e = 0; e < N; ++e) g[e] = 1.f;
        return;
    }
#pragma unroll
    for (int e = 0; e < N; e += 4) {
        const float4 v = *reinterpret_cast<const float4*>(gain + c * N + e);
        g[e] = v.x;
        g[e + 1] = v.y;
        g[e + 2] = v.z;
        g[e + 3] = v.w;
    }
}

// EB: element bytes (2 or 4); D: head_dim. NORM: also RMS-normalise the
// chunk's queries (into q_out) and keys (into the cache) on the way.
template <int EB, int D, bool NORM>
__global__ __launch_bounds__(kAppendThreads) void kv_write_kernel(
    const unsigned char* __restrict__ k_src, const unsigned char* __restrict__ v_src,
    unsigned char* __restrict__ k_pool, unsigned char* __restrict__ v_pool, int n_tok, int H,
    int64_t capacity, int64_t tok_offset, int first_blk, int n_blk, const unsigned char* q_src,
    unsigned char* q_out, const float* __restrict__ q_gain, const float* __restrict__ k_gain,
    float eps) {
    constexpr int B64 = kCacheBlock;
    constexpr int ROWB = D * EB;             // bytes of one token row of one head
    constexpr int VPR = ROWB / 16;           // 16-byte vectors per row
    constexpr int N = 16 / EB;               // elements per 16-byte vector
    constexpr int TPG = 16 / EB;             // tokens per 16-byte group of a V^T row
    constexpr int GPR = B64 / TPG;           // groups per V^T row
    constexpr int PITCH = ROWB / 4 + 1;      // LDS row pitch in 32-bit words (odd: no conflicts)
    constexpr int IT = B64 * VPR / kAppendThreads;  // 16-byte vectors per thread and tensor
    constexpr int RPI = kAppendThreads / VPR;       // rows per pass of the workgroup
    static_assert(kCacheAlign % TPG == 0, "regions must start on whole 16-byte groups");
    static_assert(64 % VPR == 0 && (B64 * VPR) % kAppendThreads == 0, "a row's lanes share a wave");
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
    const int64_t head_off = b * n_tok * src_stride + static_cast<int64_t>(h) * ROWB;
    const unsigned char* ks = k_src + head_off;
    const unsigned char* vs = v_src + head_off;
    const int64_t head = b * H + h;
    // This thread's 16-byte column of every row it visits (kAppendThreads is
    // a multiple of VPR), and its first row.
    const int c = threadIdx.x % VPR;
    const int r0 = threadIdx.x / VPR;

    float gq[N], gk[N];
    if constexpr (NORM) {
        load_gain<N>(q_gain != nullptr ? q_gain + h * D : nullptr, c, gq);
        load_gain<N>(k_gain != nullptr ? k_gain + h * D : nullptr, c, gk);
    }

    // Every load of the thread is issued before any store, so that all of
    // them are in flight together (q_out may be q itself: each element is
    // read and written by the same thread, the read first).
    uint4 kv[IT], vv[IT], qv[NORM ? IT : 1];
#pragma unroll
    for (int it = 0; it < IT; ++it) {
        const int64_t row = static_cast<int64_t>(blk) * B64 + r0 + it * RPI;
        const int64_t src = row - tok_offset;
        kv[it] = vv[it] = make_uint4(0, 0, 0, 0);
        if (NORM) qv[it] = kv[it];
        if (row >= lo && row < hi && src < n_tok) {
            kv[it] = *reinterpret_cast<const uint4*>(ks + src * src_stride + c * 16);
            vv[it] = *reinterpret_cast<const uint4*>(vs + src * src_stride + c * 16);
            if (NORM) qv[it] = *reinterpret_cast<const uint4*>(q_src + head_off + src * src_stride + c * 16);
        }
    }

    // K rows (normalised with NORM) into the cache, queries likewise into
    // q_out; V rows into LDS (zeros past the chunk's end).
#pragma unroll
    for (int it = 0; it < IT; ++it) {
        const int r = r0 + it * RPI;
        const int64_t row = static_cast<int64_t>(blk) * B64 + r;
        const bool in_block = row >= lo && row < hi;
        const int64_t src = row - tok_offset;
        const bool has_src = in_block && src < n_tok;
        if constexpr (NORM) {
            float xq[N], xk[N];
            unpack16<EB>(qv[it], xq);
            unpack16<EB>(kv[it], xk);
            rms_normalise_row<EB, D, VPR>(xq, gq, eps);
            rms_normalise_row<EB, D, VPR>(xk, gk, eps);
            kv[it] = pack16<EB>(xk);
            if (has_src) {
                const uint4 w = pack16<EB>(xq);
                store16_through(q_out + head_off + src * src_stride + c * 16, u32x4_t{w.x, w.y, w.z, w.w});
            }
        }
        if (has_src)
            store16_through(k_pool + (head * capacity + row) * ROWB + c * 16,
                            u32x4_t{kv[it].x, kv[it].y, kv[it].z, kv[it].w});
        if (in_block) {
            uint32_t* t = &tile[r * PITCH + c * 4];
            t[0] = vv[it].x;
            t[1] = vv[it].y;
            t[2] = vv[it].z;
            t[3] = vv[it].w;
        }
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
        store16_through(vblk + (static_cast<int64_t>(d) * B64 + g * TPG) * EB, u32x4_t{w[0], w[1], w[2], w[3]});
    }
}

template <int EB, int D, bool NORM>
hipError_t launch(const void* k_src, const void* v_src, void* k_pool, void* v_pool, int B,
                  int n_tok, int H, int64_t capacity, int64_t tok_offset, const void* q_src,
                  void* q_out, const float* q_gain, const float* k_gain, float eps, hipStream_t s) {
    const int64_t n_pad = (n_tok + kCacheAlign - 1) / kCacheAlign * kCacheAlign;
    const int64_t first = tok_offset / kCacheBlock;
    const int64_t last = (tok_offset + n_pad - 1) / kCacheBlock;
    const int64_t n_blk = last - first + 1;
    const int64_t grid = n_blk * B * H;
    if (grid > INT32_MAX) return hipErrorInvalidValue;
    hipLaunchKernelGGL((kv_write_kernel<EB, D, NORM>), dim3(static_cast<unsigned>(grid)),
                       dim3(kAppendThreads), 0, s, static_cast<const unsigned char*>(k_src),
                       static_cast<const unsigned char*>(v_src), static_cast<unsigned char*>(k_pool),
                       static_cast<unsigned char*>(v_pool), n_tok, H, capacity, tok_offset,
                       static_cast<int>(first), static_cast<int>(n_blk),
                       static_cast<const unsigned char*>(q_src), static_cast<unsigned char*>(q_out),
                       q_gain, k_gain, eps);
    return hipGetLastError();
}

template <bool NORM>
hipError_t dispatch(const void* k_src, const void* v_src, void* k_pool, void* v_pool, int B,
                    int n_tok, int H, int D, int elem_bytes, int64_t capacity, int64_t tok_offset,
                    const void* q_src, void* q_out, const float* q_gain, const float* k_gain,
                    float eps, hipStream_t s) {
    const int64_t n_pad = (static_cast<int64_t>(n_tok) + kCacheAlign - 1) / kCacheAlign * kCacheAlign;
    if (n_tok < 1 || tok_offset % kCacheAlign != 0 || capacity % kCacheBlock != 0 ||
        tok_offset + n_pad > capacity)
        return hipErrorInvalidValue;
#define TM_WRITE_CASE(EB_, D_)                                                                   \
    if (elem_bytes == EB_ && D == D_)                                                            \
        return launch<EB_, D_, NORM>(k_src, v_src, k_pool, v_pool, B, n_tok, H, capacity,       \
                                     tok_offset, q_src, q_out, q_gain, k_gain, eps, s);
    TM_WRITE_CASE(2, 128)
    TM_WRITE_CASE(2, 64)
    TM_WRITE_CASE(4, 128)
    TM_WRITE_CASE(4, 64)
#undef TM_WRITE_CASE
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_kv_append(const void* k_src, const void* v_src, void* k_pool, void* v_pool,
                            int B, int n_tok, int H, int D, int elem_bytes, int64_t capacity,
                            int64_t tok_offset, hipStream_t s) {
    return dispatch<false>(k_src, v_src, k_pool, v_pool, B, n_tok, H, D, elem_bytes, capacity,
                           tok_offset, nullptr, nullptr, nullptr, nullptr, 0.f, s);
}

hipError_t launch_qkv_produce(const void* q_src, const void* k_src, const void* v_src, void* q_out,
                              const float* q_gain, const float* k_gain, float eps, void* k_pool,
                              void* v_pool, int B, int n_tok, int H, int D, int elem_bytes,
                              int64_t capacity, int64_t tok_offset, hipStream_t s) {
    return dispatch<true>(k_src, v_src, k_pool, v_pool, B, n_tok, H, D, elem_bytes, capacity,
                          tok_offset, q_src, q_out, q_gain, k_gain, eps, s);
}

}  // namespace tmk
