/*
 * tm.h -- C ABI of the sparse causal streaming attention library for MI355X
 * (gfx950): the attention of the chunked autoregressive video-diffusion student
 * of TalkingMachines (arXiv 2506.03099) and the KV-cache append that lets its
 * denoising steps reuse cached context.
 *
 * The operation (paper Sec. 4.2, "Chunked Processing", "Sparse Attention
 * Pattern" and the attention equation; Sec. 4.3, "KV & Embedding Cachings"):
 * the latent sequence is a run of latent frames of T tokens each; the first R
 * frames form the starting chunk c_0 (the reference image), the following
 * frames are grouped C at a time into chunks c_1, c_2, ... (the last group may
 * be shorter). A query token of chunk c_a attends, bidirectionally, to every
 * token of c_0 and of c_{a-W} .. c_a (the paper: W = 1, i.e. c_0, c_{t-1},
 * c_t), with exact softmax(q k^T * scale) v over that key set.
 *
 * Conventions shared by every entry point
 *  - Tensors are dense, row-major, in the descriptor's dtype (fp32 or
 *    bfloat16): activations are [B, L, H, D] (batch, token, head, head_dim),
 *    i.e. token stride H*D, head stride D. Every device pointer must be
 *    16-byte aligned and point into device memory that covers the whole
 *    tensor; the library checks both before launching anything.
 *  - The caller owns all device memory and all streams. The library never
 *    allocates or frees device memory and never synchronises a stream: every
 *    launch is asynchronous on the stream passed in, so the caller orders an
 *    append before the attention that reads it (same stream, or events).
 *  - Errors: every status is TM_OK (0) or negative. All argument checks run
 *    on the host before any launch, so an error leaves caches and outputs
 *    untouched. tm_last_error() returns a thread-local message for the last
 *    failing call on that thread. No C++ exception crosses this ABI.
 *  - Threading: thread-compatible; one cache handle must not be used by two
 *    threads at once.
 */
#ifndef TM_H
#define TM_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h> /* hipStream_t */

#ifdef __cplusplus
extern "C" {
#endif

typedef enum tm_status {
    TM_OK = 0,
    TM_E_ARG = -1,      /* null/misaligned pointer, pointer not covering its tensor, bad value */
    TM_E_SHAPE = -2,    /* unsupported or inconsistent sizes */
    TM_E_DTYPE = -3,    /* unknown dtype */
    TM_E_ORDER = -4,    /* chunk index out of streaming order */
    TM_E_CAPACITY = -5, /* more tokens than the chunk (or cache) holds */
    TM_E_DEVICE = -6    /* HIP runtime reported an error */
} tm_status;

typedef enum tm_dtype { TM_F32 = 0, TM_BF16 = 1 } tm_dtype;

#define TM_MAX_WINDOW 12 /* largest supported W */

/* Problem statement of one attention layer (paper Sec. 4.2). All sizes are
 * token or frame counts, never bytes. */
typedef struct tm_attn_desc {
    int32_t batch;            /* B >= 1: independent streams processed together */
    int32_t heads;            /* H >= 1 */
    int32_t head_dim;         /* D: 64 or 128 */
    int32_t tokens_per_frame; /* T >= 1: latent tokens per latent frame */
    int32_t chunk_frames;     /* C >= 1: latent frames per chunk after c_0 */
    int32_t ref_frames;       /* R >= 1: latent frames in c_0 (reference image) */
    int32_t window;           /* W in [0, TM_MAX_WINDOW]: previous chunks seen (paper: 1) */
    int32_t dtype;            /* tm_dtype of q, k, v, o; accumulation is always fp32 */
    float softmax_scale;      /* > 0, or <= 0 for 1/sqrt(D) (the paper's 1/sqrt(d)) */
} tm_attn_desc;

/* Opaque KV cache handle: host-side bookkeeping only (descriptor, the two
 * caller-owned pools, latest chunk index, valid length of each slot). */
typedef struct tm_kv_cache tm_kv_cache;

/* Capacity of one cache in token rows per (batch, head), or 0 if the
 * descriptor is invalid. c_0 is given RC = R*T rounded up to a multiple of 8
 * rows, each of the W+1 ring slots CC = C*T rounded up to a multiple of 8, and
 * the total RC + (W+1)*CC is rounded up to a multiple of 64 (the V pool's
 * block). */
int64_t tm_kv_cache_tokens(const tm_attn_desc* desc);

/* Bytes of ONE pool (the K pool or the V pool) of one cache:
 * B * H * tm_kv_cache_tokens(desc) * D * sizeof(dtype), or 0 if invalid.
 * c_0 occupies token rows [0, R*T) and ring slot s rows [RC + s*CC, ...).
 * K pool layout: [B, H, capacity, D], i.e. each head's cached keys are one
 * contiguous run of D-element rows.
 * V pool layout: [B, H, capacity/64, D, 64]: token rows in blocks of 64, each
 * block stored dimension-major (element (row t, dim d) of a head at
 * (t/64)*64*D + d*64 + t%64), so that 8 consecutive keys of one dimension are
 * 16 contiguous bytes (the attention kernel's V^T operand). */
size_t tm_kv_cache_bytes(const tm_attn_desc* desc);

/* Create a cache over caller-allocated device pools of tm_kv_cache_bytes()
 * bytes each (16-byte aligned). The pools' contents are not read until
 * appended to. On success *out receives the handle (free it with
 * tm_kv_cache_destroy); on error *out is left unchanged. */
tm_status tm_kv_cache_create(const tm_attn_desc* desc, void* k_pool, void* v_pool,
                             tm_kv_cache** out);

/* Release the host-side handle (the pools stay the caller's). NULL is a no-op. */
void tm_kv_cache_destroy(tm_kv_cache* cache);

/* Forget every appended chunk, so the next append must be chunk 0 (a new
 * stream). Launches nothing. */
tm_status tm_kv_cache_reset(tm_kv_cache* cache);

/* Where chunk `chunk` currently lives: its first token row in the pools and
 * its valid length. TM_E_ORDER if the chunk was never appended or has been
 * evicted. Launches nothing. */
tm_status tm_kv_cache_locate(const tm_kv_cache* cache, int32_t chunk, int32_t* token_offset,
                             int32_t* n_tok);

/* Index of the latest appended chunk, or -1 for an empty cache. */
int32_t tm_kv_cache_latest(const tm_kv_cache* cache);

/* KV append / evict (paper Sec. 4.3, "KV & Embedding Cachings": the K/V of
 * c_0 and of c_{t-1} are kept so that context is never recomputed).
 * Copies the new chunk's keys and values, k and v: device [B, n_tok, H, D],
 * into the cache: chunk 0 into the c_0 rows, chunk t >= 1 into ring slot
 * (t-1) mod (W+1). Writing a slot evicts, in place, the chunk t-W-1 it held.
 * Order: the first append after create/reset must be chunk 0; afterwards
 * `chunk` must equal the latest chunk (its K/V are replaced, e.g. by the next
 * denoising step's when one cache is shared by the steps) or latest + 1
 * (advance). Otherwise TM_E_ORDER. n_tok in [1, R*T] for chunk 0 and
 * [1, C*T] for later chunks, else TM_E_CAPACITY. The bit patterns are copied
 * exactly; in the V pool the rows from n_tok up to the next multiple of 8 of
 * the chunk's region are set to zero (they are read, and masked, by the
 * attention kernel's 8-key groups). Bookkeeping is updated only when the
 * launch succeeded. */
tm_status tm_kv_append(tm_kv_cache* cache, int32_t chunk, const void* k, const void* v,
                       int32_t n_tok, hipStream_t stream);

/* Fused K/V producer: RMS normalisation of the chunk's queries and keys, and
 * the KV append, in one launch. The student keeps the attention of its
 * WAN2.1 teacher (paper Sec. 4.1), which normalises queries and keys by their
 * root mean square before the attention equation of Sec. 4.2; the keys cached
 * for later chunks (Sec. 4.3) are those normalised keys. Each (token, head)
 * row x of D elements of q and of k becomes
 *     y[d] = x[d] / sqrt(mean_d(x^2) + eps) * gain[h][d],
 * computed in fp32 and rounded to the cache dtype (nearest even for bf16).
 * q, k, v: device [B, n_tok, H, D] in the cache's dtype, as from the QKV
 * projection. q_out: device, same shape; receives the normalised queries (it
 * may be q itself, but must not otherwise overlap q, k, v or the pools).
 * q_gain, k_gain: device fp32 [H, D] (16-byte aligned), or NULL for ones.
 * eps: finite, >= 0 (TM_E_ARG otherwise). The normalised keys and the values
 * v go into the cache exactly as tm_kv_append would put k and v (same chunk
 * order rules, capacities, layouts, zero padding of V and bookkeeping): the
 * values are copied bit for bit. Replaces a separate normalisation pass and
 * tm_kv_append. */
tm_status tm_qkv_produce(tm_kv_cache* cache, int32_t chunk, const void* q, const void* k,
                         const void* v, const float* q_gain, const float* k_gain, float eps,
                         void* q_out, int32_t n_tok, hipStream_t stream);

/* Sparse causal attention forward (paper Sec. 4.2, attention equation, over
 * the key set {c_0, c_{a-W}, ..., c_a} of the query's chunk a).
 *
 * Streaming form (cache != NULL; k, v must be NULL, n_frames 0): q holds the
 * queries of the latest appended chunk, q_chunk must equal
 * tm_kv_cache_latest(cache) (else TM_E_ORDER), q is [B, n, H, D] with n that
 * chunk's appended length; every key comes from the cache (append the
 * current chunk's K/V first).
 *
 * Full-sequence form (cache == NULL): k, v are [B, n_frames*T, H, D] holding a
 * whole sequence; q_chunk = -1 means q holds all n_frames*T queries
 * (q [B, n_frames*T, H, D]); q_chunk = a >= 0 means q holds only chunk a's
 * queries (q [B, len(a), H, D]).
 *
 * o: device, same shape and dtype as q, written for every query row; it may
 * be q itself (in place) but must not otherwise overlap q, k or v.
 * lse: optional (NULL to skip) fp32 [B, H, Lq], 4-byte aligned: natural-log
 * softmax normaliser log(sum_j exp(scale * q.k_j)) of every query row.
 * Keys outside the allowed set are never read. The result is deterministic
 * (no atomics): repeated calls give identical bits. */
tm_status tm_sparse_causal_attn_fwd(const tm_attn_desc* desc, const void* q, int32_t q_chunk,
                                    const tm_kv_cache* cache, const void* k, const void* v,
                                    int32_t n_frames, void* o, float* lse, hipStream_t stream);

/* The same attention, with the output stored as fp32 instead of the
 * descriptor's dtype (paper Sec. 4.2, the attention equation; for callers
 * that keep the attention output in fp32, e.g. to add it to an fp32 residual
 * stream). Arguments, checks and launch are those of
 * tm_sparse_causal_attn_fwd, except o: device fp32 [B, Lq, H, D], 16-byte
 * aligned. For TM_BF16 inputs the arithmetic is the same kernel's, and only
 * the final rounding of O/l to bf16 (nearest even) is left out, so rounding o
 * to bf16 gives the bf16 call's output bit for bit; o then must not overlap q
 * at all. For TM_F32 inputs this is tm_sparse_causal_attn_fwd (o may be q). */
tm_status tm_sparse_causal_attn_fwd_f32out(const tm_attn_desc* desc, const void* q,
                                           int32_t q_chunk, const tm_kv_cache* cache,
                                           const void* k, const void* v, int32_t n_frames,
                                           float* o, float* lse, hipStream_t stream);

/* Backward pass of the full-sequence form (training the student through the
 * attention of Sec. 4.2): given dO = dL/dO, the gradients
 *   dV = P^T dO, dS = P * (dO V^T - rowsum(dO * O)), dQ = scale dS K,
 *   dK = scale dS^T Q,
 * with P the masked row softmax recomputed from lse. Only allowed (query, key)
 * pairs are visited (the same tile skipping as the forward).
 * q, k, v, o, dout: device bf16 [B, L, H, D] with L = n_frames * T, as in the
 * full-sequence forward with q_chunk = -1 (o is its output).
 * lse: device fp32 [B, H, L], the forward's natural-log normaliser (4-byte
 * aligned). delta: caller-owned device fp32 workspace [B, H, L], overwritten
 * with rowsum(dO * O). dq, dk, dv: device bf16 [B, L, H, D], every row
 * written; they must not overlap each other or any input.
 * TM_BF16 only (else TM_E_DTYPE). Three launches on `stream`; deterministic
 * (no atomics). */
tm_status tm_sparse_causal_attn_bwd(const tm_attn_desc* desc, int32_t n_frames, const void* q,
                                    const void* k, const void* v, const void* o, const float* lse,
                                    const void* dout, float* delta, void* dq, void* dk, void* dv,
                                    hipStream_t stream);

/* The same backward pass without the caller's workspace, for callers that
 * cannot allocate device memory (code under HIP graph capture, serving loops
 * or harnesses that forbid allocation): delta lives in a device-global array
 * of the library, 8 MiB per GPU (room for B * H * L <= 2^21 rows), which each
 * GPU the library runs on holds until the process ends. Arguments, checks,
 * launches and results are those of tm_sparse_causal_attn_bwd without delta;
 * B * H * L above 2^21 returns TM_E_CAPACITY. The call allocates nothing.
 * Every call on one GPU uses that GPU's one array (each call writes delta
 * before reading it): calls that overlap in time on one GPU, on different
 * streams or from different threads, race and give wrong gradients; order
 * them. */
tm_status tm_sparse_causal_attn_bwd_noalloc(const tm_attn_desc* desc, int32_t n_frames,
                                            const void* q, const void* k, const void* v,
                                            const void* o, const float* lse, const void* dout,
                                            void* dq, void* dk, void* dv, hipStream_t stream);

/* Number of allowed (query, key) pairs per (batch, head) of the call the same
 * arguments would make (4*D of FLOPs each); -1 on invalid arguments. Pure host
 * arithmetic, launches nothing; the streaming form reads the cache
 * bookkeeping. */
int64_t tm_allowed_pairs(const tm_attn_desc* desc, int32_t q_chunk, const tm_kv_cache* cache,
                         int32_t n_frames);

/* Audio cross-attention with a local frame window and a face mask (paper
 * Sec. 4.1: "Audio Cross Attention with Attention Mask", "Audio Projection
 * Layer", "Speaking/Silence Mode"). Audio tokens are aligned to latent frames,
 * A per frame, covering frames 0 .. F_a - 1; each face has its own audio
 * stream (a silent face's stream holds the special embedding's keys and
 * values). A query token of latent frame f whose face id is m in [0, M)
 * attends, with exact softmax(q k^T * scale) v, to the audio tokens of stream
 * m in frames max(0, f - w) .. min(F_a - 1, f + w) (w = 2: five frames centred
 * on f); a token with any other face id (-1: no face) gets a zero output. */
#define TM_MAX_AUDIO_STREAMS 32

typedef struct tm_audio_desc {
    int32_t batch;            /* B >= 1 */
    int32_t heads;            /* H >= 1 */
    int32_t head_dim;         /* D: 64 or 128 */
    int32_t tokens_per_frame; /* T >= 1: query tokens per latent frame */
    int32_t audio_per_frame;  /* A >= 1: audio tokens per latent frame */
    int32_t audio_frames;     /* F_a >= 1: latent frames the audio covers */
    int32_t streams;          /* M in [1, TM_MAX_AUDIO_STREAMS]: audio streams (faces) */
    int32_t half_window;      /* w >= 0 (paper: 2, a window of five frames) */
    int32_t dtype;            /* TM_BF16 only; accumulation is fp32 */
    float softmax_scale;      /* > 0, or <= 0 for 1/sqrt(D) */
} tm_audio_desc;

/* q: device [B, n_tok, H, D], query row i in latent frame
 * first_frame + i / T; every frame of the run must lie inside the audio
 * (first_frame + ceil(n_tok / T) <= F_a, else TM_E_SHAPE).
 * ak, av: device [B, M, F_a * A, H, D] audio keys and values.
 * face: device int32 [B, n_tok] (4-byte aligned), the stream of each query
 * token; ids outside [0, M) mean no face.
 * o: device [B, n_tok, H, D], every row written; may be q itself (in place)
 * but must not otherwise overlap q, ak, av or face.
 * A frame's window (at most (2w + 1) * A keys, rounded up to 32) must fit in
 * one workgroup's LDS: at most 288 keys at D = 128, 608 at D = 64, else
 * TM_E_SHAPE. n_tok = 0 launches nothing. P is rounded to bf16 before P V;
 * the row sums add the fp32 P. The result is deterministic. */
tm_status tm_audio_cross_attn_fwd(const tm_audio_desc* desc, const void* q, int32_t first_frame,
                                  int32_t n_tok, const void* ak, const void* av,
                                  const int32_t* face, void* o, hipStream_t stream);

/* The same audio cross-attention with the output stored as fp32 (paper
 * Sec. 4.1; for callers that keep the cross-attention output in fp32):
 * arguments and checks as tm_audio_cross_attn_fwd, except o: device fp32
 * [B, n_tok, H, D], 16-byte aligned, not overlapping q. The arithmetic is the
 * bf16 call's; only the final rounding to bf16 (nearest even) is left out,
 * so rounding o to bf16 gives that call's output bit for bit. Rows without a
 * face get zeros. */
tm_status tm_audio_cross_attn_fwd_f32out(const tm_audio_desc* desc, const void* q,
                                         int32_t first_frame, int32_t n_tok, const void* ak,
                                         const void* av, const int32_t* face, float* o,
                                         hipStream_t stream);

/* Message of the last failing call on this thread ("" if none). */
const char* tm_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* TM_H */
