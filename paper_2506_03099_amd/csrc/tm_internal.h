// Internal interface between the host-side API (tm_api.cpp) and the HIP
// kernels (attn_fwd.hip, kv_append.hip, audio_attn.hip). Not part of the
// public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tmk {

constexpr int kMaxRanges = 16;  // key ranges of one query segment (>= TM_MAX_WINDOW + 2)

// Rows per query tile of each attention kernel; the host needs them to count
// tiles per chunk.
constexpr int kTileRowsBf16 = 256;
constexpr int kTileRowsF32 = 64;

// KV-cache pools are organised in blocks of this many token rows. The V pool
// stores each block dimension-major: [D][kCacheBlock] per (batch, head, block),
// so that the attention kernel's V^T operand is a contiguous 16-byte read.
constexpr int kCacheBlock = 64;
// Cache regions (c_0 and every ring slot) start on multiples of this many
// tokens, so that every 16-byte group of a V block row belongs to one region.
constexpr int kCacheAlign = 8;

// One attention launch. Element strides (not bytes) for batch, token and head.
// With v_blocked != 0, v is a cache V pool: element (token t, dim d) of a head
// sits at (t / 64) * 64 * D + d * 64 + t % 64 from the head's base, v_st is
// unused, and every key range starts on a multiple of kCacheAlign.
struct AttnArgs {
    const void* q;
    const void* k;
    const void* v;
    void* o;
    float* lse;  // [B, H, Lq] or null
    int64_t q_sb, q_st, q_sh;
    int64_t k_sb, k_st, k_sh;
    int64_t v_sb, v_st, v_sh;
    int64_t o_sb, o_st, o_sh;
    int32_t o_f32;  // bf16 kernel: store O as fp32 (the values before the final rounding)
    int32_t v_blocked;
    int32_t B, H, Lq;
    float scale_log2;  // softmax scale * log2(e)
    int32_t n_qtiles;  // query tiles per (batch, head)
    // mode 0: every query row of the buffer belongs to one chunk and sees the
    //         same key ranges (streaming form, or one chunk of a sequence);
    // mode 1: the buffer holds a whole sequence (row i = position i); each
    //         tile's chunk and key ranges follow from the geometry below.
    int32_t mode;
    int32_t n_ranges;  // mode 0
    int32_t range_begin[kMaxRanges];
    int32_t range_end[kMaxRanges];
    int32_t ref_tok;      // mode 1: R*T (clipped to the sequence)
    int32_t chunk_tok;    // mode 1: C*T
    int32_t window;       // mode 1: W
    int32_t seq_len;      // mode 1: tokens in the sequence
    int32_t ref_tiles;    // mode 1: query tiles of c_0
    int32_t chunk_tiles;  // mode 1: query tiles of a full chunk
};

hipError_t launch_attn_bf16(const AttnArgs& a, int head_dim, hipStream_t s);
hipError_t launch_attn_f32(const AttnArgs& a, int head_dim, hipStream_t s);

// Copy n_tok tokens of K and V from [B, n_tok, H, D] into the cache pools at
// token row `tok_offset` (a multiple of kCacheAlign): K into [B, H, capacity,
// D], V into [B, H, capacity / 64, D, 64]. The V columns from n_tok up to the
// next multiple of kCacheAlign are written as zeros. `capacity` is a multiple
// of kCacheBlock; elem_bytes is 2 or 4.
hipError_t launch_kv_append(const void* k_src, const void* v_src, void* k_pool, void* v_pool,
                            int B, int n_tok, int H, int D, int elem_bytes, int64_t capacity,
                            int64_t tok_offset, hipStream_t s);

// The same write of the chunk's V, while the chunk's queries (into q_out, same
// layout as q_src) and keys (into the K pool) are RMS-normalised per (token,
// head) row over D: x / sqrt(mean(x^2) + eps) * gain[h, :] (gain NULL: ones),
// in fp32, rounded to the element type. q_out may equal q_src.
hipError_t launch_qkv_produce(const void* q_src, const void* k_src, const void* v_src, void* q_out,
                              const float* q_gain, const float* k_gain, float eps, void* k_pool,
                              void* v_pool, int B, int n_tok, int H, int D, int elem_bytes,
                              int64_t capacity, int64_t tok_offset, hipStream_t s);

// Audio cross-attention of a run of latent-frame tokens (bf16). q, o: [B, n,
// H, D]; ak, av: [B, M, La, H, D] with La = F_a * A; face: [B, n] stream index
// per query token (ids outside [0, M) mean no face: zero output).
struct AudioArgs {
    const void* q;
    const void* ak;
    const void* av;
    const int32_t* face;
    void* o;
    int32_t B, n, H, M, La;
    int32_t T;             // query tokens per latent frame
    int32_t A;             // audio tokens per latent frame
    int32_t first_frame;   // latent frame of query row 0
    int32_t half_window;   // frames f - w .. f + w
    int32_t n_frames;      // latent frames the n rows span
    int32_t parts;         // workgroups per (batch, head, frame)
    int32_t max_keys_pad;  // most window keys of any frame, rounded up to 32
    int32_t o_f32;         // store o as fp32 (the values before the final rounding)
    float scale_log2;      // softmax scale * log2(e)
    int32_t n_cwg;         // compute workgroups (B * H * n_frames * parts); set by the launcher
    int32_t zrows;         // token rows per zero-fill workgroup; set by the launcher
    int32_t q_stage;       // queries (and bf16 output rows) staged in LDS; set by the launcher
};

// Most 32-row blocks of one frame per audio workgroup: a frame with more
// blocks is split over several workgroups, which take every parts-th block.
constexpr int kAudioBlocksPerPart = 64;

// LDS of one audio workgroup: a window of nk_pad keys as K rows and V rows of
// D bf16 each, then one word per wave (8), the face waves' row counts per
// segment (32), the count of one stream's rows (one word, padded to 16 bytes)
// and those rows compacted (16-bit indices). Staging the queries and the
// output through LDS adds one slot of 32 rows of D bf16 per wave.
constexpr size_t kAudioFaceLds = 4 * 8 + 4 * 32 + 16 + 2 * 32 * kAudioBlocksPerPart;
__host__ __device__ constexpr size_t audio_lds_bytes(int head_dim, int nk_pad) {
    return 2 * static_cast<size_t>(nk_pad) * head_dim * 2 + kAudioFaceLds;
}
__host__ __device__ constexpr size_t audio_stage_lds_bytes(int head_dim) {
    return static_cast<size_t>(8) * 32 * head_dim * 2;
}
constexpr size_t kAudioMaxLds = 160 * 1024;  // gfx950: 160 KiB of LDS per workgroup
// Most window keys (a multiple of 32) that fit: 288 at D = 128, 608 at D = 64.
template <int D>
constexpr int kAudioMaxKeys = static_cast<int>((kAudioMaxLds - kAudioFaceLds) / (2 * 2 * D)) / 32 * 32;

hipError_t launch_audio_attn_bf16(const AudioArgs& a, int head_dim, hipStream_t s);

// Backward of the whole-sequence attention (bf16): q, k, v, o, dout, dq, dk,
// dv are [B, L, H, D]; lse (natural log) and delta (written here) are fp32
// [B, H, L]. Query tiles of kBwdQTile rows and key tiles of kBwdKTile keys
// never straddle a chunk: ref tiles for c_0, then chunk tiles per chunk.
constexpr int kBwdQTile = 128;
constexpr int kBwdKTile = 128;
struct BwdArgs {
    const void* q;
    const void* k;
    const void* v;
    const void* o;
    const float* lse;
    const void* dout;
    float* delta;
    void* dq;
    void* dk;
    void* dv;
    int32_t B, H, L;
    int32_t ref_tok, chunk_tok, window;  // R*T, C*T, W
    float scale, scale_log2;
    int32_t q_tiles, q_ref_tiles, q_chunk_tiles;
    int32_t k_tiles, k_ref_tiles, k_chunk_tiles;
};
hipError_t launch_attn_bwd_bf16(const BwdArgs& a, int head_dim, hipStream_t s);

// The device-global workspace of the allocation-free backward: room for delta
// of B * H * L <= kBwdScratchFloats rows (8 MiB per GPU). bwd_scratch_address
// returns its address on the current device (looked up on the first call per
// device); kernels get that address, never the symbol.
constexpr int64_t kBwdScratchFloats = int64_t(1) << 21;
hipError_t bwd_scratch_address(float** out);

}  // namespace tmk
