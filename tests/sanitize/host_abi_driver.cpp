// Driver of the C ABI (include/tm.h) for the sanitizer build: tm_api.cpp is
// compiled with AddressSanitizer and UndefinedBehaviorSanitizer (host code
// only) into this executable, which links the kernels from libtm.so. Every
// host path of the ABI runs here: descriptor and argument validation, the cache
// size arithmetic, the key-range planner's pair counts (closed forms of the
// chunk pattern, TalkingMachines Sec. 4.2), the limits of every size, and with
// --gpu the cache bookkeeping, appends, forward, backward and audio calls on
// real device memory. Exit status 0 and "host ABI driver: all checks passed"
// when every check holds; a sanitizer report aborts the run.
#include <hip/hip_runtime.h>

#include <climits>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "tm.h"

namespace {

int g_failed = 0;
int g_checks = 0;

#define EXPECT(cond)                                                                       \
    do {                                                                                   \
        ++g_checks;                                                                        \
        if (!(cond)) {                                                                     \
            ++g_failed;                                                                    \
            std::fprintf(stderr, "FAILED %s:%d: %s (last error: %s)\n", __FILE__, __LINE__, \
                         #cond, tm_last_error());                                          \
        }                                                                                  \
    } while (0)

// Aligned, non-null, and not memory the HIP runtime knows.
void* const FAKE = reinterpret_cast<void*>(uintptr_t(1) << 40);
void* fake(uintptr_t off) { return reinterpret_cast<void*>((uintptr_t(1) << 40) + off); }

tm_attn_desc desc(int32_t B = 1, int32_t H = 40, int32_t D = 128, int32_t T = 1560, int32_t C = 3,
                  int32_t R = 1, int32_t W = 1, int32_t dtype = TM_BF16, float scale = 0.f) {
    tm_attn_desc d;
    d.batch = B;
    d.heads = H;
    d.head_dim = D;
    d.tokens_per_frame = T;
    d.chunk_frames = C;
    d.ref_frames = R;
    d.window = W;
    d.dtype = dtype;
    d.softmax_scale = scale;
    return d;
}

tm_audio_desc adesc(int32_t A = 32, int32_t Fa = 21, int32_t M = 1, int32_t w = 2,
                    int32_t D = 128, int32_t dtype = TM_BF16) {
    tm_audio_desc d;
    d.batch = 1;
    d.heads = 40;
    d.head_dim = D;
    d.tokens_per_frame = 1560;
    d.audio_per_frame = A;
    d.audio_frames = Fa;
    d.streams = M;
    d.half_window = w;
    d.dtype = dtype;
    d.softmax_scale = 0.f;
    return d;
}

// Allowed pairs of a whole sequence by brute force over chunk indices (the
// rule of Sec. 4.2: a query of chunk a sees c_0 and chunks a-W .. a).
int64_t brute_pairs(int64_t frames, int64_t T, int64_t C, int64_t R, int64_t W) {
    const int64_t L = frames * T;
    std::vector<int64_t> chunk(L);
    for (int64_t p = 0; p < L; ++p) {
        const int64_t f = p / T;
        chunk[p] = f < R ? 0 : 1 + (f - R) / C;
    }
    int64_t n = 0;
    for (int64_t i = 0; i < L; ++i)
        for (int64_t j = 0; j < L; ++j)
            n += chunk[j] == 0 || (chunk[j] >= chunk[i] - W && chunk[j] <= chunk[i]);
    return n;
}

void host_checks() {
    // cache sizes: c_0 and each slot rounded up to 8 rows, the total to 64
    tm_attn_desc d = desc();
    EXPECT(tm_kv_cache_tokens(&d) == 10944);
    EXPECT(tm_kv_cache_bytes(&d) == size_t(40) * 10944 * 128 * 2);
    tm_attn_desc d2 = desc(2, 40, 128, 3600, 3, 1, 3, TM_F32);
    EXPECT(tm_kv_cache_tokens(&d2) == 46848);
    tm_attn_desc d3 = desc(1, 40, 128, 7, 10, 3, 12);
    EXPECT(tm_kv_cache_tokens(&d3) == 960);

    // invalid descriptors have no size; extreme values must not overflow
    const tm_attn_desc bad[] = {desc(1, 40, 96), desc(0), desc(1, 0), desc(1, 40, 128, 0),
                                desc(1, 40, 128, 1560, 0), desc(1, 40, 128, 1560, 3, 0),
                                desc(1, 40, 128, 1560, 3, 1, -1), desc(1, 40, 128, 1560, 3, 1, 13),
                                desc(1, 40, 128, 1560, 3, 1, 1, 7),
                                desc(1, 40, 128, INT32_MAX, INT32_MAX, INT32_MAX, 12),
                                desc(INT32_MAX, INT32_MAX), desc(1, 40, 128, INT32_MAX, 1, 1, 12)};
    for (const tm_attn_desc& b : bad) {
        EXPECT(tm_kv_cache_bytes(&b) == 0);
        EXPECT(tm_kv_cache_tokens(&b) == 0);
    }
    EXPECT(tm_kv_cache_bytes(nullptr) == 0);
    tm_attn_desc nan_scale = desc();
    nan_scale.softmax_scale = NAN;
    EXPECT(tm_allowed_pairs(&nan_scale, -1, nullptr, 21) == -1);

    // planner: closed forms and brute force
    EXPECT(tm_allowed_pairs(&d, -1, nullptr, 21) == 316368000);
    tm_attn_desc lit = desc(1, 40, 128, 1560, 3, 3, 1);
    EXPECT(tm_allowed_pairs(&lit, -1, nullptr, 21) == 394243200);
    tm_attn_desc tiny = desc(1, 2, 64, 64, 2, 1, 1, TM_F32);
    EXPECT(tm_allowed_pairs(&tiny, -1, nullptr, 9) == 151552);
    EXPECT(tm_allowed_pairs(&tiny, 2, nullptr, 9) == 128 * 320);
    EXPECT(tm_allowed_pairs(&tiny, 5, nullptr, 9) == -1);
    EXPECT(tm_allowed_pairs(&tiny, -2, nullptr, 9) == -1);
    EXPECT(tm_allowed_pairs(&tiny, -1, nullptr, 0) == -1);
    EXPECT(tm_allowed_pairs(&tiny, -1, nullptr, INT32_MAX) == -1);  // more than 2^30 tokens
    const int geo[][5] = {{13, 7, 2, 1, 0}, {13, 7, 2, 2, 3}, {5, 11, 4, 1, 1}, {2, 5, 3, 3, 1},
                          {30, 3, 1, 1, 12}, {9, 1, 1, 1, 12}};
    for (const auto& g : geo) {
        tm_attn_desc dg = desc(1, 1, 64, g[1], g[2], g[3], g[4]);
        EXPECT(tm_allowed_pairs(&dg, -1, nullptr, g[0]) == brute_pairs(g[0], g[1], g[2], g[3], g[4]));
    }

    // forward argument checks
    EXPECT(tm_sparse_causal_attn_fwd(nullptr, FAKE, -1, nullptr, FAKE, FAKE, 21, FAKE, nullptr,
                                     nullptr) == TM_E_ARG);
    tm_attn_desc hd = desc(1, 40, 96);
    EXPECT(tm_sparse_causal_attn_fwd(&hd, FAKE, -1, nullptr, FAKE, FAKE, 21, FAKE, nullptr,
                                     nullptr) == TM_E_SHAPE);
    tm_attn_desc dt = desc(1, 40, 128, 1560, 3, 1, 1, 5);
    EXPECT(tm_sparse_causal_attn_fwd(&dt, FAKE, -1, nullptr, FAKE, FAKE, 21, FAKE, nullptr,
                                     nullptr) == TM_E_DTYPE);
    EXPECT(tm_sparse_causal_attn_fwd(&d, FAKE, 8, nullptr, FAKE, FAKE, 21, FAKE, nullptr,
                                     nullptr) == TM_E_SHAPE);
    EXPECT(tm_sparse_causal_attn_fwd(&d, nullptr, -1, nullptr, FAKE, FAKE, 21, FAKE, nullptr,
                                     nullptr) == TM_E_ARG);
    EXPECT(tm_sparse_causal_attn_fwd(&d, FAKE, -1, nullptr, fake(8), FAKE, 21, FAKE, nullptr,
                                     nullptr) == TM_E_ARG);
    EXPECT(tm_sparse_causal_attn_fwd(&d, FAKE, -1, nullptr, FAKE, FAKE, 21, FAKE, nullptr,
                                     nullptr) == TM_E_ARG);
    EXPECT(tm_sparse_causal_attn_fwd_f32out(&d, FAKE, -1, nullptr, FAKE, FAKE, 21,
                                            static_cast<float*>(FAKE), nullptr, nullptr) == TM_E_ARG);
    EXPECT(std::strlen(tm_last_error()) > 0);

    // cache handle checks
    tm_kv_cache* h = nullptr;
    EXPECT(tm_kv_cache_create(&d, FAKE, FAKE, &h) == TM_E_ARG);  // the same pool twice
    EXPECT(tm_kv_cache_create(&d, FAKE, fake(uintptr_t(1) << 32), &h) == TM_E_ARG);
    EXPECT(h == nullptr);
    EXPECT(tm_kv_cache_create(nullptr, FAKE, FAKE, &h) == TM_E_ARG);
    EXPECT(tm_kv_cache_create(&d, FAKE, fake(uintptr_t(1) << 32), nullptr) == TM_E_ARG);
    EXPECT(tm_kv_cache_reset(nullptr) == TM_E_ARG);
    EXPECT(tm_kv_cache_latest(nullptr) == -1);
    int32_t off = 0, n = 0;
    EXPECT(tm_kv_cache_locate(nullptr, 0, &off, &n) == TM_E_ARG);
    tm_kv_cache_destroy(nullptr);
    EXPECT(tm_kv_append(nullptr, 0, FAKE, FAKE, 10, nullptr) == TM_E_ARG);
    EXPECT(tm_qkv_produce(nullptr, 0, FAKE, FAKE, FAKE, nullptr, nullptr, 0.f, FAKE, 10, nullptr) ==
           TM_E_ARG);
    EXPECT(tm_qkv_produce(nullptr, 0, nullptr, FAKE, FAKE, nullptr, nullptr, 0.f, FAKE, 10, nullptr) ==
           TM_E_ARG);

    // backward argument checks
    tm_attn_desc f32 = desc(1, 40, 128, 1560, 3, 1, 1, TM_F32);
    float* F = static_cast<float*>(FAKE);
    EXPECT(tm_sparse_causal_attn_bwd(&f32, 21, FAKE, FAKE, FAKE, FAKE, F, FAKE, F, FAKE, FAKE,
                                     FAKE, nullptr) == TM_E_DTYPE);
    EXPECT(tm_sparse_causal_attn_bwd(&d, 0, FAKE, FAKE, FAKE, FAKE, F, FAKE, F, FAKE, FAKE, FAKE,
                                     nullptr) == TM_E_SHAPE);
    EXPECT(tm_sparse_causal_attn_bwd(&d, 21, FAKE, FAKE, FAKE, FAKE, F, FAKE, nullptr, FAKE, FAKE,
                                     FAKE, nullptr) == TM_E_ARG);
    EXPECT(tm_sparse_causal_attn_bwd(&d, INT32_MAX, FAKE, FAKE, FAKE, FAKE, F, FAKE, F, FAKE, FAKE,
                                     FAKE, nullptr) == TM_E_SHAPE);
    EXPECT(tm_sparse_causal_attn_bwd(&d, 21, FAKE, FAKE, FAKE, FAKE, F, FAKE, F, FAKE, FAKE, FAKE,
                                     nullptr) == TM_E_ARG);
    tm_attn_desc wide = desc(1, 64, 64, 1024);
    EXPECT(tm_sparse_causal_attn_bwd_noalloc(&wide, 33, FAKE, FAKE, FAKE, FAKE, F, FAKE, FAKE, FAKE,
                                             FAKE, nullptr) == TM_E_CAPACITY);
    EXPECT(tm_sparse_causal_attn_bwd_noalloc(&wide, 32, FAKE, FAKE, FAKE, FAKE, F, FAKE, FAKE, FAKE,
                                             FAKE, nullptr) == TM_E_ARG);

    // audio argument checks
    tm_audio_desc a = adesc();
    const int32_t* face = static_cast<const int32_t*>(FAKE);
    EXPECT(tm_audio_cross_attn_fwd(nullptr, FAKE, 0, 10, FAKE, FAKE, face, FAKE, nullptr) == TM_E_ARG);
    EXPECT(tm_audio_cross_attn_fwd(&a, FAKE, 0, 0, FAKE, FAKE, face, FAKE, nullptr) == TM_OK);
    EXPECT(tm_audio_cross_attn_fwd(&a, FAKE, -1, 10, FAKE, FAKE, face, FAKE, nullptr) == TM_E_SHAPE);
    EXPECT(tm_audio_cross_attn_fwd(&a, FAKE, 19, 3 * 1560, FAKE, FAKE, face, FAKE, nullptr) ==
           TM_E_SHAPE);
    EXPECT(tm_audio_cross_attn_fwd(&a, FAKE, 18, 3 * 1560, FAKE, FAKE, face, FAKE, nullptr) ==
           TM_E_ARG);
    tm_audio_desc big = adesc(58);  // frame 2 sees frames 0..4: 5 * 58 = 290 > 288 keys
    EXPECT(tm_audio_cross_attn_fwd(&big, FAKE, 0, 3 * 1560, FAKE, FAKE, face, FAKE, nullptr) ==
           TM_E_SHAPE);
    EXPECT(tm_audio_cross_attn_fwd(&big, FAKE, 0, 10, FAKE, FAKE, face, FAKE, nullptr) ==
           TM_E_ARG);  // frame 0 alone: its window is clipped to 3 * 58 = 174 keys
    tm_audio_desc huge = adesc(INT32_MAX, INT32_MAX, 1, INT32_MAX);
    EXPECT(tm_audio_cross_attn_fwd(&huge, FAKE, 0, 10, FAKE, FAKE, face, FAKE, nullptr) == TM_E_SHAPE);
    tm_audio_desc ad = adesc(32, 21, 1, 2, 128, TM_F32);
    EXPECT(tm_audio_cross_attn_fwd(&ad, FAKE, 0, 10, FAKE, FAKE, face, FAKE, nullptr) == TM_E_DTYPE);
    EXPECT(tm_audio_cross_attn_fwd_f32out(&a, FAKE, 0, 10, FAKE, FAKE, face,
                                          static_cast<float*>(FAKE), nullptr) == TM_E_ARG);
}

#define HIP_OK(x) EXPECT((x) == hipSuccess)

// Device paths: the cache's bookkeeping through appends, overwrites, eviction
// and reset; forward calls of both forms and both output types; the backward
// with and without workspace; the audio kernel. The results are checked by
// the GPU parity tests; here every status and every piece of bookkeeping is.
void gpu_checks() {
    const int B = 1, H = 2, D = 64, T = 16, C = 2, R = 1, W = 1;
    tm_attn_desc d = desc(B, H, D, T, C, R, W, TM_BF16);
    const size_t pool = tm_kv_cache_bytes(&d);
    void *kp = nullptr, *vp = nullptr, *q = nullptr, *k = nullptr, *v = nullptr, *o = nullptr;
    float *lse = nullptr, *of = nullptr;
    const size_t chunk_bytes = size_t(B) * C * T * H * D * 2;
    HIP_OK(hipMalloc(&kp, pool));
    HIP_OK(hipMalloc(&vp, pool));
    HIP_OK(hipMalloc(&q, chunk_bytes));
    HIP_OK(hipMalloc(&k, chunk_bytes));
    HIP_OK(hipMalloc(&v, chunk_bytes));
    HIP_OK(hipMalloc(&o, chunk_bytes));
    HIP_OK(hipMalloc(&of, chunk_bytes * 2));
    HIP_OK(hipMalloc(&lse, size_t(B) * H * C * T * 4));
    HIP_OK(hipMemset(q, 0, chunk_bytes));
    HIP_OK(hipMemset(k, 0, chunk_bytes));
    HIP_OK(hipMemset(v, 0, chunk_bytes));
    tm_kv_cache* c = nullptr;
    EXPECT(tm_kv_cache_create(&d, kp, vp, &c) == TM_OK);
    EXPECT(c != nullptr && tm_kv_cache_latest(c) == -1);
    EXPECT(tm_kv_append(c, 1, k, v, C * T, nullptr) == TM_E_ORDER);  // chunk 0 first
    EXPECT(tm_kv_append(c, 0, k, v, R * T + 1, nullptr) == TM_E_CAPACITY);
    EXPECT(tm_kv_append(c, 0, k, v, 0, nullptr) == TM_E_SHAPE);
    EXPECT(tm_kv_append(c, 0, k, v, R * T, nullptr) == TM_OK);
    EXPECT(tm_kv_append(c, 2, k, v, C * T, nullptr) == TM_E_ORDER);  // skips chunk 1
    int32_t off = -1, n = -1;
    for (int t = 1; t <= 4; ++t) {
        EXPECT(tm_kv_append(c, t, k, v, t == 4 ? C * T - 5 : C * T, nullptr) == TM_OK);
        EXPECT(tm_kv_append(c, t, k, v, C * T, nullptr) == TM_OK);  // the next step overwrites
        EXPECT(tm_kv_cache_latest(c) == t);
        EXPECT(tm_kv_cache_locate(c, t, &off, &n) == TM_OK && n == C * T);
        if (t >= 3) EXPECT(tm_kv_cache_locate(c, t - 2, &off, &n) == TM_E_ORDER);  // evicted
        EXPECT(tm_sparse_causal_attn_fwd(&d, q, t, c, nullptr, nullptr, 0, o, lse, nullptr) == TM_OK);
        EXPECT(tm_sparse_causal_attn_fwd_f32out(&d, q, t, c, nullptr, nullptr, 0, of, nullptr,
                                                nullptr) == TM_OK);
        EXPECT(tm_sparse_causal_attn_fwd(&d, q, t - 1, c, nullptr, nullptr, 0, o, nullptr,
                                         nullptr) == TM_E_ORDER);
        EXPECT(tm_allowed_pairs(&d, t, c, 0) == int64_t(C * T) * (R * T + (t == 1 ? 1 : 2) * C * T));
    }
    EXPECT(tm_kv_cache_locate(c, 0, &off, &n) == TM_OK && off == 0 && n == R * T);
    // o may be q only with the same element type
    EXPECT(tm_sparse_causal_attn_fwd(&d, q, 4, c, nullptr, nullptr, 0, q, nullptr, nullptr) == TM_OK);
    EXPECT(tm_sparse_causal_attn_fwd_f32out(&d, q, 4, c, nullptr, nullptr, 0,
                                            static_cast<float*>(q), nullptr, nullptr) == TM_E_ARG);
    EXPECT(tm_kv_cache_reset(c) == TM_OK && tm_kv_cache_latest(c) == -1);
    EXPECT(tm_kv_append(c, 1, k, v, C * T, nullptr) == TM_E_ORDER);
    tm_kv_cache_destroy(c);

    // full-sequence forward and backward over 5 frames (80 tokens)
    const int frames = 5, L = frames * T;
    const size_t seq = size_t(B) * L * H * D * 2;
    void *sq, *sk, *sv, *so, *sdo, *dq, *dk, *dv;
    float *slse, *delta;
    for (void** p : {&sq, &sk, &sv, &so, &sdo, &dq, &dk, &dv}) {
        HIP_OK(hipMalloc(p, seq));
        HIP_OK(hipMemset(*p, 0, seq));
    }
    HIP_OK(hipMalloc(&slse, size_t(B) * H * L * 4));
    HIP_OK(hipMalloc(&delta, size_t(B) * H * L * 4));
    EXPECT(tm_sparse_causal_attn_fwd(&d, sq, -1, nullptr, sk, sv, frames, so, slse, nullptr) == TM_OK);
    EXPECT(tm_sparse_causal_attn_fwd(&d, sq, -1, nullptr, sk, sv, frames + 1, so, slse, nullptr) ==
           TM_E_ARG);  // the tensors are too short for 6 frames
    EXPECT(tm_sparse_causal_attn_bwd(&d, frames, sq, sk, sv, so, slse, sdo, delta, dq, dk, dv,
                                     nullptr) == TM_OK);
    EXPECT(tm_sparse_causal_attn_bwd_noalloc(&d, frames, sq, sk, sv, so, slse, sdo, dq, dk, dv,
                                             nullptr) == TM_OK);
    EXPECT(tm_sparse_causal_attn_bwd(&d, frames, sq, sk, sv, so, slse, sdo, delta, sq, dk, dv,
                                     nullptr) == TM_E_ARG);  // dq overlaps q

    // audio: one frame of 16 tokens, 4 audio tokens per frame, 3 frames of audio
    tm_audio_desc a = adesc(4, 3, 1, 2, D);
    a.heads = H;
    a.tokens_per_frame = T;
    void *ak, *av;
    int32_t* face;
    const size_t abytes = size_t(B) * 1 * 3 * 4 * H * D * 2;
    HIP_OK(hipMalloc(&ak, abytes));
    HIP_OK(hipMalloc(&av, abytes));
    HIP_OK(hipMalloc(reinterpret_cast<void**>(&face), size_t(T) * 4));
    HIP_OK(hipMemset(ak, 0, abytes));
    HIP_OK(hipMemset(av, 0, abytes));
    HIP_OK(hipMemset(face, 0, size_t(T) * 4));
    EXPECT(tm_audio_cross_attn_fwd(&a, sq, 1, T, ak, av, face, so, nullptr) == TM_OK);
    EXPECT(tm_audio_cross_attn_fwd_f32out(&a, sq, 1, T, ak, av, face, of, nullptr) == TM_OK);
    HIP_OK(hipDeviceSynchronize());

    for (void* p : {kp, vp, q, k, v, o, static_cast<void*>(of), static_cast<void*>(lse), sq, sk, sv,
                    so, sdo, dq, dk, dv, static_cast<void*>(slse), static_cast<void*>(delta), ak, av,
                    static_cast<void*>(face)})
        HIP_OK(hipFree(p));
}

}  // namespace

int main(int argc, char** argv) {
    const bool gpu = argc > 1 && std::strcmp(argv[1], "--gpu") == 0;
    host_checks();
    if (gpu) gpu_checks();
    std::printf("host ABI driver (%s): %d checks, %d failed\n", gpu ? "host + gpu" : "host",
                g_checks, g_failed);
    if (g_failed == 0) std::printf("host ABI driver: all checks passed\n");
    return g_failed == 0 ? 0 : 1;
}
