// Host side of the C ABI declared in include/tm.h: argument validation, KV
// cache bookkeeping, the key-range planner and kernel launches.
//
// Key-range planning (TalkingMachines, Sec. 4.2, "Chunked Processing" and
// "Sparse Attention Pattern"): a query of chunk a may see c_0 and the chunks
// a-W .. a. In a whole sequence those keys form at most two contiguous
// position ranges, [0, R*T) and [start(max(1, a-W)), end(a)), which merge into
// one when a-W <= 1. In the cache (Sec. 4.3, "KV & Embedding Cachings") c_0
// sits in front of a ring of W+1 chunk slots, chunk t >= 1 in slot
// (t-1) mod (W+1); when the latest chunk is t, every cached chunk is in the
// window of t, so the keys are the valid rows of c_0 and of each filled slot,
// merged into contiguous ranges. Regions start on multiples of 8 tokens and
// the pools hold a multiple of 64 token rows (the V pool's block size).

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <string>
#include <utility>
#include <vector>

#include "tm.h"
#include "tm_internal.h"

struct tm_kv_cache {
    tm_attn_desc desc;
    void* k_pool;
    void* v_pool;
    int32_t latest;  // -1: empty
    int32_t ref_len;
    int32_t slot_chunk[TM_MAX_WINDOW + 1];  // chunk held by each ring slot, -1: none
    int32_t slot_len[TM_MAX_WINDOW + 1];
};

namespace {

thread_local std::string g_err;

tm_status fail(tm_status st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
    return st;
}

struct Geo {
    int64_t B, H, D, T, C, R, W;
    int dtype;
    size_t elem;
    float scale;
    int64_t RT, CT;          // tokens of c_0 and of a full chunk
    int64_t ref_cap, slot_cap;  // cache rows reserved for c_0 and for each ring slot
    int64_t capacity;        // cache rows per (batch, head)
};

int64_t round_up(int64_t a, int64_t b) { return (a + b - 1) / b * b; }

constexpr int64_t kMaxTokens = int64_t(1) << 30;

tm_status check_desc(const tm_attn_desc* d, Geo* g) {
    if (d == nullptr) return fail(TM_E_ARG, "descriptor is NULL");
    if (d->dtype != TM_F32 && d->dtype != TM_BF16)
        return fail(TM_E_DTYPE, "dtype %d is neither TM_F32 nor TM_BF16", d->dtype);
    if (d->batch < 1 || d->heads < 1) return fail(TM_E_SHAPE, "batch and heads must be >= 1");
    if (d->head_dim != 64 && d->head_dim != 128)
        return fail(TM_E_SHAPE, "head_dim %d unsupported (64 or 128)", d->head_dim);
    if (d->tokens_per_frame < 1 || d->chunk_frames < 1 || d->ref_frames < 1)
        return fail(TM_E_SHAPE, "tokens_per_frame, chunk_frames and ref_frames must be >= 1");
    if (d->window < 0 || d->window > TM_MAX_WINDOW)
        return fail(TM_E_SHAPE, "window %d outside [0, %d]", d->window, TM_MAX_WINDOW);
    if (!std::isfinite(d->softmax_scale))
        return fail(TM_E_ARG, "softmax_scale is not finite");
    g->B = d->batch;
    g->H = d->heads;
    g->D = d->head_dim;
    g->T = d->tokens_per_frame;
    g->C = d->chunk_frames;
    g->R = d->ref_frames;
    g->W = d->window;
    g->dtype = d->dtype;
    g->elem = d->dtype == TM_BF16 ? 2 : 4;
    g->scale = d->softmax_scale > 0.f ? d->softmax_scale : 1.f / std::sqrt(float(d->head_dim));
    g->RT = g->R * g->T;  // each factor < 2^31: no overflow in 64 bits
    g->CT = g->C * g->T;
    if (g->RT > kMaxTokens || g->CT > kMaxTokens)  // before any product of them
        return fail(TM_E_SHAPE, "chunk too large (more than 2^30 tokens)");
    g->ref_cap = round_up(g->RT, tmk::kCacheAlign);
    g->slot_cap = round_up(g->CT, tmk::kCacheAlign);
    g->capacity = round_up(g->ref_cap + (g->W + 1) * g->slot_cap, tmk::kCacheBlock);
    if (g->capacity > kMaxTokens)
        return fail(TM_E_SHAPE, "cache too large (more than 2^30 tokens)");
    if (g->B * g->H > (int64_t(1) << 20)) return fail(TM_E_SHAPE, "batch * heads too large");
    return TM_OK;
}

// The pointer must be a 16-byte (or `align`-byte) aligned device pointer of
// the current device whose allocation covers `bytes` bytes from it.
tm_status check_ptr(const void* p, size_t bytes, const char* name, size_t align = 16) {
    if (p == nullptr) return fail(TM_E_ARG, "%s is NULL", name);
    if (reinterpret_cast<uintptr_t>(p) % align != 0)
        return fail(TM_E_ARG, "%s is not %zu-byte aligned", name, align);
    hipPointerAttribute_t attr;
    if (hipPointerGetAttributes(&attr, p) != hipSuccess) {
        (void)hipGetLastError();
        return fail(TM_E_ARG, "%s is not a pointer known to the HIP runtime", name);
    }
    if (attr.type != hipMemoryTypeDevice && attr.type != hipMemoryTypeManaged)
        return fail(TM_E_ARG, "%s is not device memory", name);
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) {
        (void)hipGetLastError();
        return fail(TM_E_DEVICE, "hipGetDevice failed");
    }
    if (attr.device != dev)
        return fail(TM_E_ARG, "%s lives on device %d, current device is %d", name, attr.device, dev);
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    if (hipMemGetAddressRange(&base, &size, const_cast<void*>(p)) != hipSuccess) {
        (void)hipGetLastError();
        return fail(TM_E_ARG, "%s: allocation bounds unknown", name);
    }
    const uintptr_t b = reinterpret_cast<uintptr_t>(base), q = reinterpret_cast<uintptr_t>(p);
    if (q < b || q - b > size || bytes > size - (q - b))
        return fail(TM_E_ARG, "%s: %zu bytes from it run past the end of its allocation", name,
                    bytes);
    return TM_OK;
}

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return x < y + nb && y < x + na;
}

// ---- chunk geometry of a whole sequence of L tokens
int64_t chunk_start(const Geo& g, int64_t c) { return c == 0 ? 0 : g.RT + (c - 1) * g.CT; }
int64_t chunk_end(const Geo& g, int64_t c, int64_t L) {
    return std::min(c == 0 ? g.RT : g.RT + c * g.CT, L);
}
int64_t n_chunks(const Geo& g, int64_t L) {
    return L <= g.RT ? 1 : 1 + (L - g.RT + g.CT - 1) / g.CT;
}
int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

struct Plan {
    int mode = 0;
    int64_t Lq = 0;
    std::vector<std::pair<int64_t, int64_t>> ranges;  // mode 0
    int64_t seq_len = 0;                              // mode 1
    int64_t pairs = 0;                                // allowed pairs per (b, h)
};

// Keys of query chunk a in a sequence of L tokens, as merged ranges.
std::vector<std::pair<int64_t, int64_t>> sequence_ranges(const Geo& g, int64_t a, int64_t L) {
    if (a == 0) return {{0, std::min(g.RT, L)}};
    const int64_t lo = std::max<int64_t>(1, a - g.W);
    if (lo == 1) return {{0, chunk_end(g, a, L)}};
    return {{0, g.RT}, {chunk_start(g, lo), chunk_end(g, a, L)}};
}

int64_t range_len(const std::vector<std::pair<int64_t, int64_t>>& r) {
    int64_t n = 0;
    for (const auto& x : r) n += x.second - x.first;
    return n;
}

tm_status plan_sequence(const Geo& g, int32_t n_frames, int32_t q_chunk, Plan* p) {
    if (n_frames < 1) return fail(TM_E_SHAPE, "n_frames must be >= 1");
    const int64_t L = int64_t(n_frames) * g.T;
    if (L > kMaxTokens) return fail(TM_E_SHAPE, "sequence too long");
    const int64_t nc = n_chunks(g, L);
    if (q_chunk < -1 || q_chunk >= nc)
        return fail(TM_E_SHAPE, "q_chunk %d outside [-1, %lld)", q_chunk, (long long)nc);
    p->seq_len = L;
    if (q_chunk == -1) {
        p->mode = 1;
        p->Lq = L;
        p->pairs = 0;
        for (int64_t a = 0; a < nc; ++a)
            p->pairs += (chunk_end(g, a, L) - chunk_start(g, a)) * range_len(sequence_ranges(g, a, L));
    } else {
        p->mode = 0;
        p->Lq = chunk_end(g, q_chunk, L) - chunk_start(g, q_chunk);
        p->ranges = sequence_ranges(g, q_chunk, L);
        p->pairs = p->Lq * range_len(p->ranges);
    }
    return TM_OK;
}

tm_status plan_stream(const Geo& g, const tm_kv_cache* c, Plan* p) {
    const int32_t t = c->latest;
    std::vector<std::pair<int64_t, int64_t>> r;
    r.push_back({0, c->ref_len});
    int64_t lq = c->ref_len;
    for (int64_t ch = std::max<int64_t>(1, t - g.W); ch <= t; ++ch) {
        const int slot = int((ch - 1) % (g.W + 1));
        if (c->slot_chunk[slot] != ch) return fail(TM_E_ORDER, "chunk %lld missing from the cache", (long long)ch);
        const int64_t b = g.ref_cap + slot * g.slot_cap;
        r.push_back({b, b + c->slot_len[slot]});
        if (ch == t) lq = c->slot_len[slot];
    }
    std::sort(r.begin(), r.end());
    std::vector<std::pair<int64_t, int64_t>> m;
    for (const auto& x : r) {
        if (!m.empty() && m.back().second == x.first) m.back().second = x.second;
        else m.push_back(x);
    }
    p->mode = 0;
    p->Lq = lq;
    p->ranges = m;
    p->pairs = lq * range_len(m);
    return TM_OK;
}

bool same_desc(const tm_attn_desc& a, const tm_attn_desc& b) {
    return a.batch == b.batch && a.heads == b.heads && a.head_dim == b.head_dim &&
           a.tokens_per_frame == b.tokens_per_frame && a.chunk_frames == b.chunk_frames &&
           a.ref_frames == b.ref_frames && a.window == b.window && a.dtype == b.dtype &&
           a.softmax_scale == b.softmax_scale;
}

// Resolve the call's plan (shared by the forward and tm_allowed_pairs).
tm_status make_plan(const tm_attn_desc* desc, int32_t q_chunk, const tm_kv_cache* cache,
                    int32_t n_frames, Geo* g, Plan* p) {
    tm_status st = check_desc(desc, g);
    if (st != TM_OK) return st;
    if (cache != nullptr) {
        if (n_frames != 0) return fail(TM_E_ARG, "streaming form takes n_frames = 0");
        if (!same_desc(cache->desc, *desc))
            return fail(TM_E_ARG, "descriptor differs from the one the cache was created with");
        if (cache->latest < 0) return fail(TM_E_ORDER, "the cache is empty");
        if (q_chunk != cache->latest)
            return fail(TM_E_ORDER, "q_chunk %d is not the latest appended chunk %d", q_chunk,
                        cache->latest);
        return plan_stream(*g, cache, p);
    }
    return plan_sequence(*g, n_frames, q_chunk, p);
}

}  // namespace

extern "C" {

int64_t tm_kv_cache_tokens(const tm_attn_desc* desc) {
    Geo g;
    if (check_desc(desc, &g) != TM_OK) return 0;
    return g.capacity;
}

size_t tm_kv_cache_bytes(const tm_attn_desc* desc) {
    Geo g;
    if (check_desc(desc, &g) != TM_OK) return 0;
    return size_t(g.B) * size_t(g.H) * size_t(g.capacity) * size_t(g.D) * g.elem;
}

tm_status tm_kv_cache_create(const tm_attn_desc* desc, void* k_pool, void* v_pool,
                             tm_kv_cache** out) {
    Geo g;
    tm_status st = check_desc(desc, &g);
    if (st != TM_OK) return st;
    if (out == nullptr) return fail(TM_E_ARG, "out is NULL");
    const size_t bytes = tm_kv_cache_bytes(desc);
    if (k_pool == v_pool || overlaps(k_pool, bytes, v_pool, bytes))
        return fail(TM_E_ARG, "k_pool and v_pool overlap");
    if ((st = check_ptr(k_pool, bytes, "k_pool")) != TM_OK) return st;
    if ((st = check_ptr(v_pool, bytes, "v_pool")) != TM_OK) return st;
    tm_kv_cache* c = new (std::nothrow) tm_kv_cache;
    if (c == nullptr) return fail(TM_E_ARG, "out of host memory");
    c->desc = *desc;
    c->k_pool = k_pool;
    c->v_pool = v_pool;
    tm_kv_cache_reset(c);
    *out = c;
    return TM_OK;
}

void tm_kv_cache_destroy(tm_kv_cache* cache) { delete cache; }

tm_status tm_kv_cache_reset(tm_kv_cache* cache) {
    if (cache == nullptr) return fail(TM_E_ARG, "cache is NULL");
    cache->latest = -1;
    cache->ref_len = 0;
    for (int i = 0; i <= TM_MAX_WINDOW; ++i) {
        cache->slot_chunk[i] = -1;
        cache->slot_len[i] = 0;
    }
    return TM_OK;
}

int32_t tm_kv_cache_latest(const tm_kv_cache* cache) { return cache ? cache->latest : -1; }

tm_status tm_kv_cache_locate(const tm_kv_cache* cache, int32_t chunk, int32_t* token_offset,
                             int32_t* n_tok) {
    if (cache == nullptr || token_offset == nullptr || n_tok == nullptr)
        return fail(TM_E_ARG, "NULL argument");
    if (chunk < 0 || cache->latest < 0 || chunk > cache->latest)
        return fail(TM_E_ORDER, "chunk %d not in the cache", chunk);
    Geo g;
    if (check_desc(&cache->desc, &g) != TM_OK) return TM_E_ARG;
    const tm_attn_desc& d = cache->desc;
    if (chunk == 0) {
        *token_offset = 0;
        *n_tok = cache->ref_len;
        return TM_OK;
    }
    const int slot = (chunk - 1) % (d.window + 1);
    if (cache->slot_chunk[slot] != chunk) return fail(TM_E_ORDER, "chunk %d was evicted", chunk);
    *token_offset = int32_t(g.ref_cap + slot * g.slot_cap);
    *n_tok = cache->slot_len[slot];
    return TM_OK;
}

namespace {

// Shared by tm_kv_append and tm_qkv_produce: order and capacity rules, pointer
// checks, the launch, and the bookkeeping (updated only after a successful
// launch). With q != nullptr the chunk's queries and keys are RMS-normalised
// on the way (queries into q_out).
tm_status write_chunk(tm_kv_cache* cache, int32_t chunk, const void* q, const void* k,
                      const void* v, const float* q_gain, const float* k_gain, float eps,
                      void* q_out, int32_t n_tok, hipStream_t stream) {
    if (cache == nullptr) return fail(TM_E_ARG, "cache is NULL");
    Geo g;
    tm_status st = check_desc(&cache->desc, &g);
    if (st != TM_OK) return st;
    if (cache->latest < 0 ? chunk != 0 : (chunk != cache->latest && chunk != cache->latest + 1))
        return fail(TM_E_ORDER, "chunk %d cannot follow latest chunk %d", chunk, cache->latest);
    const int64_t cap = chunk == 0 ? g.RT : g.CT;
    if (n_tok < 1) return fail(TM_E_SHAPE, "n_tok must be >= 1");
    if (n_tok > cap)
        return fail(TM_E_CAPACITY, "n_tok %d exceeds the %s of %lld tokens", n_tok,
                    chunk == 0 ? "reference chunk" : "chunk", (long long)cap);
    const size_t bytes = size_t(g.B) * size_t(n_tok) * size_t(g.H) * size_t(g.D) * g.elem;
    const size_t pool_bytes = tm_kv_cache_bytes(&cache->desc);
    if ((st = check_ptr(k, bytes, "k")) != TM_OK) return st;
    if ((st = check_ptr(v, bytes, "v")) != TM_OK) return st;
    if (overlaps(k, bytes, cache->k_pool, pool_bytes) || overlaps(k, bytes, cache->v_pool, pool_bytes) ||
        overlaps(v, bytes, cache->k_pool, pool_bytes) || overlaps(v, bytes, cache->v_pool, pool_bytes))
        return fail(TM_E_ARG, "k/v overlap the cache pools");
    if ((st = check_ptr(cache->k_pool, pool_bytes, "k_pool")) != TM_OK) return st;
    if ((st = check_ptr(cache->v_pool, pool_bytes, "v_pool")) != TM_OK) return st;
    if (q != nullptr) {
        if (!std::isfinite(eps) || eps < 0.f) return fail(TM_E_ARG, "eps must be finite and >= 0");
        if ((st = check_ptr(q, bytes, "q")) != TM_OK) return st;
        if ((st = check_ptr(q_out, bytes, "q_out")) != TM_OK) return st;
        if (q_out != q && overlaps(q_out, bytes, q, bytes))
            return fail(TM_E_ARG, "q_out overlaps q without being q");
        if (overlaps(q_out, bytes, k, bytes) || overlaps(q_out, bytes, v, bytes) ||
            overlaps(q_out, bytes, cache->k_pool, pool_bytes) ||
            overlaps(q_out, bytes, cache->v_pool, pool_bytes))
            return fail(TM_E_ARG, "q_out overlaps k, v or the cache pools");
        const size_t gain_bytes = size_t(g.H) * size_t(g.D) * sizeof(float);
        if (q_gain != nullptr && (st = check_ptr(q_gain, gain_bytes, "q_gain", 16)) != TM_OK) return st;
        if (k_gain != nullptr && (st = check_ptr(k_gain, gain_bytes, "k_gain", 16)) != TM_OK) return st;
    }
    const int slot = chunk == 0 ? -1 : int((chunk - 1) % (g.W + 1));
    const int64_t offset = chunk == 0 ? 0 : g.ref_cap + slot * g.slot_cap;
    const hipError_t e =
        q == nullptr
            ? tmk::launch_kv_append(k, v, cache->k_pool, cache->v_pool, int(g.B), n_tok, int(g.H),
                                    int(g.D), int(g.elem), g.capacity, offset, stream)
            : tmk::launch_qkv_produce(q, k, v, q_out, q_gain, k_gain, eps, cache->k_pool,
                                      cache->v_pool, int(g.B), n_tok, int(g.H), int(g.D),
                                      int(g.elem), g.capacity, offset, stream);
    if (e != hipSuccess)
        return fail(TM_E_DEVICE, "%s launch: %s", q == nullptr ? "kv_append" : "qkv_produce",
                    hipGetErrorString(e));
    if (chunk == 0) {
        tm_kv_cache_reset(cache);
        cache->ref_len = n_tok;
    } else {
        cache->slot_chunk[slot] = chunk;
        cache->slot_len[slot] = n_tok;
    }
    cache->latest = chunk;
    return TM_OK;
}

}  // namespace

tm_status tm_kv_append(tm_kv_cache* cache, int32_t chunk, const void* k, const void* v,
                       int32_t n_tok, hipStream_t stream) {
    return write_chunk(cache, chunk, nullptr, k, v, nullptr, nullptr, 0.f, nullptr, n_tok, stream);
}

tm_status tm_qkv_produce(tm_kv_cache* cache, int32_t chunk, const void* q, const void* k,
                         const void* v, const float* q_gain, const float* k_gain, float eps,
                         void* q_out, int32_t n_tok, hipStream_t stream) {
    if (q == nullptr) return fail(TM_E_ARG, "q is NULL");
    return write_chunk(cache, chunk, q, k, v, q_gain, k_gain, eps, q_out, n_tok, stream);
}

int64_t tm_allowed_pairs(const tm_attn_desc* desc, int32_t q_chunk, const tm_kv_cache* cache,
                         int32_t n_frames) {
    Geo g;
    Plan p;
    if (make_plan(desc, q_chunk, cache, n_frames, &g, &p) != TM_OK) return -1;
    return p.pairs;
}

}  // extern "C"

namespace {

// The forward of both output types: o holds elements of the descriptor's
// dtype, or fp32 when o_f32 is set (for bf16 inputs the values before the
// final rounding; for fp32 inputs the same call).
tm_status attn_fwd(const tm_attn_desc* desc, const void* q, int32_t q_chunk,
                   const tm_kv_cache* cache, const void* k, const void* v, int32_t n_frames,
                   void* o, bool o_f32, float* lse, hipStream_t stream) {
    Geo g;
    Plan p;
    tm_status st = make_plan(desc, q_chunk, cache, n_frames, &g, &p);
    if (st != TM_OK) return st;

    tmk::AttnArgs a{};
    const int64_t HD = g.H * g.D;
    size_t kv_bytes;
    if (cache != nullptr) {
        if (k != nullptr || v != nullptr) return fail(TM_E_ARG, "streaming form takes k = v = NULL");
        a.k = cache->k_pool;
        a.v = cache->v_pool;
        a.k_sb = a.v_sb = g.H * g.capacity * g.D;
        a.k_sh = a.v_sh = g.capacity * g.D;
        a.k_st = g.D;
        a.v_st = 0;
        a.v_blocked = 1;
        kv_bytes = tm_kv_cache_bytes(desc);
    } else {
        a.k = k;
        a.v = v;
        a.k_sb = a.v_sb = p.seq_len * HD;
        a.k_sh = a.v_sh = g.D;
        a.k_st = a.v_st = HD;
        kv_bytes = size_t(g.B) * size_t(p.seq_len) * size_t(HD) * g.elem;
    }
    const size_t q_bytes = size_t(g.B) * size_t(p.Lq) * size_t(HD) * g.elem;
    const size_t o_bytes = size_t(g.B) * size_t(p.Lq) * size_t(HD) * (o_f32 ? 4 : g.elem);
    const size_t lse_bytes = size_t(g.B) * size_t(g.H) * size_t(p.Lq) * sizeof(float);
    if ((st = check_ptr(q, q_bytes, "q")) != TM_OK) return st;
    if ((st = check_ptr(a.k, kv_bytes, cache ? "k_pool" : "k")) != TM_OK) return st;
    if ((st = check_ptr(a.v, kv_bytes, cache ? "v_pool" : "v")) != TM_OK) return st;
    if ((st = check_ptr(o, o_bytes, "o")) != TM_OK) return st;
    if (lse != nullptr && (st = check_ptr(lse, lse_bytes, "lse", 4)) != TM_OK) return st;
    if (overlaps(o, o_bytes, a.k, kv_bytes) || overlaps(o, o_bytes, a.v, kv_bytes))
        return fail(TM_E_ARG, "o overlaps k or v");
    // In place (o == q) only when o and q have the same element type.
    if ((o != q || o_bytes != q_bytes) && overlaps(o, o_bytes, q, q_bytes))
        return fail(TM_E_ARG, "o overlaps q (only o == q with the same dtype is allowed)");
    if (lse != nullptr && (overlaps(lse, lse_bytes, a.k, kv_bytes) ||
                           overlaps(lse, lse_bytes, a.v, kv_bytes) ||
                           overlaps(lse, lse_bytes, q, q_bytes) || overlaps(lse, lse_bytes, o, o_bytes)))
        return fail(TM_E_ARG, "lse overlaps another tensor");

    a.q = q;
    a.o = o;
    a.o_f32 = o_f32 && g.dtype == TM_BF16;
    a.lse = lse;
    a.q_sb = a.o_sb = p.Lq * HD;
    a.q_st = a.o_st = HD;
    a.q_sh = a.o_sh = g.D;
    a.B = int32_t(g.B);
    a.H = int32_t(g.H);
    a.Lq = int32_t(p.Lq);
    a.scale_log2 = float(double(g.scale) * 1.4426950408889634);
    a.mode = p.mode;
    const int64_t BM = g.dtype == TM_BF16 ? tmk::kTileRowsBf16 : tmk::kTileRowsF32;
    int64_t tiles;
    if (p.mode == 0) {
        if (p.ranges.size() > size_t(tmk::kMaxRanges))
            return fail(TM_E_SHAPE, "too many key ranges (%zu)", p.ranges.size());
        a.n_ranges = int32_t(p.ranges.size());
        for (size_t i = 0; i < p.ranges.size(); ++i) {
            a.range_begin[i] = int32_t(p.ranges[i].first);
            a.range_end[i] = int32_t(p.ranges[i].second);
        }
        tiles = ceil_div(p.Lq, BM);
    } else {
        const int64_t L = p.seq_len, nc = n_chunks(g, L);
        a.ref_tok = int32_t(std::min(g.RT, L));
        a.chunk_tok = int32_t(g.CT);
        a.window = int32_t(g.W);
        a.seq_len = int32_t(L);
        a.ref_tiles = int32_t(ceil_div(a.ref_tok, BM));
        a.chunk_tiles = int32_t(ceil_div(g.CT, BM));
        tiles = a.ref_tiles;
        if (nc >= 2) {
            tiles += (nc - 2) * a.chunk_tiles;
            tiles += ceil_div(chunk_end(g, nc - 1, L) - chunk_start(g, nc - 1), BM);
        }
    }
    if (tiles * g.B * g.H > INT32_MAX) return fail(TM_E_SHAPE, "grid too large");
    a.n_qtiles = int32_t(tiles);

    const hipError_t e = g.dtype == TM_BF16 ? tmk::launch_attn_bf16(a, int(g.D), stream)
                                            : tmk::launch_attn_f32(a, int(g.D), stream);
    if (e != hipSuccess) return fail(TM_E_DEVICE, "attention launch: %s", hipGetErrorString(e));
    return TM_OK;
}

}  // namespace

extern "C" {

tm_status tm_sparse_causal_attn_fwd(const tm_attn_desc* desc, const void* q, int32_t q_chunk,
                                    const tm_kv_cache* cache, const void* k, const void* v,
                                    int32_t n_frames, void* o, float* lse, hipStream_t stream) {
    return attn_fwd(desc, q, q_chunk, cache, k, v, n_frames, o, false, lse, stream);
}

tm_status tm_sparse_causal_attn_fwd_f32out(const tm_attn_desc* desc, const void* q,
                                           int32_t q_chunk, const tm_kv_cache* cache,
                                           const void* k, const void* v, int32_t n_frames,
                                           float* o, float* lse, hipStream_t stream) {
    return attn_fwd(desc, q, q_chunk, cache, k, v, n_frames, o, true, lse, stream);
}

}  // extern "C"

namespace {

// The backward with a caller's delta workspace, or (delta == nullptr) with the
// library's device-global workspace, which allocates nothing.
tm_status attn_bwd(const tm_attn_desc* desc, int32_t n_frames, const void* q, const void* k,
                   const void* v, const void* o, const float* lse, const void* dout, float* delta,
                   void* dq, void* dk, void* dv, hipStream_t stream) {
    const bool use_scratch = delta == nullptr;
    Geo g;
    tm_status st = check_desc(desc, &g);
    if (st != TM_OK) return st;
    if (g.dtype != TM_BF16) return fail(TM_E_DTYPE, "the backward pass runs in TM_BF16 only");
    if (n_frames < 1) return fail(TM_E_SHAPE, "n_frames must be >= 1");
    const int64_t L = int64_t(n_frames) * g.T;
    if (L > kMaxTokens) return fail(TM_E_SHAPE, "sequence too long (more than 2^30 tokens)");
    if (use_scratch && g.B * g.H * L > tmk::kBwdScratchFloats)
        return fail(TM_E_CAPACITY,
                    "batch * heads * tokens = %lld exceeds the %lld rows of the library's "
                    "workspace; use tm_sparse_causal_attn_bwd with a caller-owned delta",
                    static_cast<long long>(g.B * g.H * L),
                    static_cast<long long>(tmk::kBwdScratchFloats));
    const size_t t_bytes = size_t(g.B) * size_t(L) * size_t(g.H) * size_t(g.D) * 2;
    const size_t r_bytes = size_t(g.B) * size_t(g.H) * size_t(L) * sizeof(float);
    const void* ins[] = {q, k, v, o, dout};
    const char* in_names[] = {"q", "k", "v", "o", "dO"};
    for (int i = 0; i < 5; ++i)
        if ((st = check_ptr(ins[i], t_bytes, in_names[i])) != TM_OK) return st;
    if ((st = check_ptr(lse, r_bytes, "lse", 4)) != TM_OK) return st;
    if (!use_scratch && (st = check_ptr(delta, r_bytes, "delta", 4)) != TM_OK) return st;
    void* outs[] = {dq, dk, dv};
    const char* out_names[] = {"dq", "dk", "dv"};
    for (int i = 0; i < 3; ++i) {
        if ((st = check_ptr(outs[i], t_bytes, out_names[i])) != TM_OK) return st;
        for (int j = 0; j < 5; ++j)
            if (overlaps(outs[i], t_bytes, ins[j], t_bytes))
                return fail(TM_E_ARG, "%s overlaps %s", out_names[i], in_names[j]);
        if (overlaps(outs[i], t_bytes, lse, r_bytes) ||
            (!use_scratch && overlaps(outs[i], t_bytes, delta, r_bytes)))
            return fail(TM_E_ARG, "%s overlaps lse or delta", out_names[i]);
        for (int j = 0; j < i; ++j)
            if (overlaps(outs[i], t_bytes, outs[j], t_bytes))
                return fail(TM_E_ARG, "%s overlaps %s", out_names[i], out_names[j]);
    }
    if (!use_scratch) {
        for (int j = 0; j < 5; ++j)
            if (overlaps(delta, r_bytes, ins[j], t_bytes))
                return fail(TM_E_ARG, "delta overlaps %s", in_names[j]);
        if (overlaps(delta, r_bytes, lse, r_bytes)) return fail(TM_E_ARG, "delta overlaps lse");
    } else {
        const hipError_t e = tmk::bwd_scratch_address(&delta);
        if (e != hipSuccess)
            return fail(TM_E_DEVICE, "workspace address: %s", hipGetErrorString(e));
    }

    tmk::BwdArgs a{};
    a.q = q;
    a.k = k;
    a.v = v;
    a.o = o;
    a.lse = lse;
    a.dout = dout;
    a.delta = delta;
    a.dq = dq;
    a.dk = dk;
    a.dv = dv;
    a.B = int32_t(g.B);
    a.H = int32_t(g.H);
    a.L = int32_t(L);
    a.ref_tok = int32_t(g.RT);
    a.chunk_tok = int32_t(g.CT);
    a.window = int32_t(g.W);
    a.scale = g.scale;
    a.scale_log2 = float(double(g.scale) * 1.4426950408889634);
    const int64_t nc = n_chunks(g, L);
    const int64_t ref_rows = std::min(g.RT, L);
    const int64_t qrt = ceil_div(ref_rows, tmk::kBwdQTile), qct = ceil_div(g.CT, tmk::kBwdQTile);
    const int64_t krt = ceil_div(ref_rows, tmk::kBwdKTile), kct = ceil_div(g.CT, tmk::kBwdKTile);
    const int64_t q_tiles = qrt + (nc - 1) * qct, k_tiles = krt + (nc - 1) * kct;
    if (q_tiles * g.B * g.H > INT32_MAX || k_tiles * g.B * g.H > INT32_MAX)
        return fail(TM_E_SHAPE, "grid too large");
    a.q_tiles = int32_t(q_tiles);
    a.q_ref_tiles = int32_t(qrt);
    a.q_chunk_tiles = int32_t(qct);
    a.k_tiles = int32_t(k_tiles);
    a.k_ref_tiles = int32_t(krt);
    a.k_chunk_tiles = int32_t(kct);
    const hipError_t e = tmk::launch_attn_bwd_bf16(a, int(g.D), stream);
    if (e != hipSuccess) return fail(TM_E_DEVICE, "backward launch: %s", hipGetErrorString(e));
    return TM_OK;
}

}  // namespace

extern "C" {

tm_status tm_sparse_causal_attn_bwd(const tm_attn_desc* desc, int32_t n_frames, const void* q,
                                    const void* k, const void* v, const void* o, const float* lse,
                                    const void* dout, float* delta, void* dq, void* dk, void* dv,
                                    hipStream_t stream) {
    if (delta == nullptr) return fail(TM_E_ARG, "delta is NULL");
    return attn_bwd(desc, n_frames, q, k, v, o, lse, dout, delta, dq, dk, dv, stream);
}

tm_status tm_sparse_causal_attn_bwd_noalloc(const tm_attn_desc* desc, int32_t n_frames,
                                            const void* q, const void* k, const void* v,
                                            const void* o, const float* lse, const void* dout,
                                            void* dq, void* dk, void* dv, hipStream_t stream) {
    return attn_bwd(desc, n_frames, q, k, v, o, lse, dout, nullptr, dq, dk, dv, stream);
}

}  // extern "C"

namespace {

tm_status audio_fwd(const tm_audio_desc* d, const void* q, int32_t first_frame, int32_t n_tok,
                    const void* ak, const void* av, const int32_t* face, void* o, bool o_f32,
                    hipStream_t stream) {
    if (d == nullptr) return fail(TM_E_ARG, "descriptor is NULL");
    if (d->dtype != TM_BF16) return fail(TM_E_DTYPE, "audio cross-attention runs in TM_BF16 only");
    if (d->batch < 1 || d->heads < 1) return fail(TM_E_SHAPE, "batch and heads must be >= 1");
    if (int64_t(d->batch) * d->heads > (int64_t(1) << 20))
        return fail(TM_E_SHAPE, "batch * heads too large");
    if (d->head_dim != 64 && d->head_dim != 128)
        return fail(TM_E_SHAPE, "head_dim %d unsupported (64 or 128)", d->head_dim);
    if (d->tokens_per_frame < 1 || d->audio_per_frame < 1 || d->audio_frames < 1)
        return fail(TM_E_SHAPE, "tokens_per_frame, audio_per_frame and audio_frames must be >= 1");
    if (d->streams < 1 || d->streams > TM_MAX_AUDIO_STREAMS)
        return fail(TM_E_SHAPE, "streams %d outside [1, %d]", d->streams, TM_MAX_AUDIO_STREAMS);
    if (d->half_window < 0) return fail(TM_E_SHAPE, "half_window must be >= 0");
    if (!std::isfinite(d->softmax_scale)) return fail(TM_E_ARG, "softmax_scale is not finite");
    const int64_t La = int64_t(d->audio_frames) * d->audio_per_frame;
    if (La > kMaxTokens) return fail(TM_E_SHAPE, "audio too long (more than 2^30 tokens)");
    if (n_tok < 0 || first_frame < 0) return fail(TM_E_SHAPE, "n_tok and first_frame must be >= 0");
    if (n_tok == 0) return TM_OK;  // nothing to attend
    const int64_t T = d->tokens_per_frame;
    const int64_t n_frames = ceil_div(n_tok, T);
    if (int64_t(first_frame) + n_frames > d->audio_frames)
        return fail(TM_E_SHAPE, "query frames %d..%lld lie past the audio's %d frames", first_frame,
                    static_cast<long long>(first_frame + n_frames - 1), d->audio_frames);
    // The widest window of the run's frames must fit the workgroup's LDS.
    int64_t max_keys = 0;
    for (int64_t f = first_frame; f < first_frame + n_frames; ++f) {
        const int64_t lo = std::max<int64_t>(0, f - d->half_window);
        const int64_t hi = std::min<int64_t>(d->audio_frames - 1, f + d->half_window);
        max_keys = std::max(max_keys, (hi - lo + 1) * d->audio_per_frame);
    }
    if (max_keys > kMaxTokens) return fail(TM_E_SHAPE, "audio window too long");
    const int64_t keys_pad = round_up(max_keys, 32);
    if (tmk::audio_lds_bytes(d->head_dim, int(keys_pad)) > tmk::kAudioMaxLds)
        return fail(TM_E_SHAPE, "audio window of %lld keys does not fit in LDS (at most %d keys at D = %d)",
                    static_cast<long long>(max_keys), d->head_dim == 128 ? 288 : 608, d->head_dim);

    const size_t HD = size_t(d->heads) * size_t(d->head_dim);
    const size_t q_bytes = size_t(d->batch) * size_t(n_tok) * HD * 2;
    const size_t o_bytes = size_t(d->batch) * size_t(n_tok) * HD * (o_f32 ? 4 : 2);
    const size_t a_bytes = size_t(d->batch) * size_t(d->streams) * size_t(La) * HD * 2;
    const size_t f_bytes = size_t(d->batch) * size_t(n_tok) * sizeof(int32_t);
    tm_status st;
    if ((st = check_ptr(q, q_bytes, "q")) != TM_OK) return st;
    if ((st = check_ptr(ak, a_bytes, "ak")) != TM_OK) return st;
    if ((st = check_ptr(av, a_bytes, "av")) != TM_OK) return st;
    if ((st = check_ptr(face, f_bytes, "face", 4)) != TM_OK) return st;
    if ((st = check_ptr(o, o_bytes, "o")) != TM_OK) return st;
    if (overlaps(o, o_bytes, ak, a_bytes) || overlaps(o, o_bytes, av, a_bytes) ||
        overlaps(o, o_bytes, face, f_bytes))
        return fail(TM_E_ARG, "o overlaps ak, av or face");
    if ((o != q || o_f32) && overlaps(o, o_bytes, q, q_bytes))
        return fail(TM_E_ARG, "o overlaps q (only o == q with the same dtype is allowed)");

    const int64_t rows_per_frame = std::min<int64_t>(T, n_tok);
    const int64_t blocks = ceil_div(rows_per_frame, 32);
    const int64_t parts = ceil_div(blocks, tmk::kAudioBlocksPerPart);
    if (int64_t(d->batch) * d->heads * n_frames * parts > INT32_MAX)
        return fail(TM_E_SHAPE, "grid too large");
    tmk::AudioArgs a{};
    a.q = q;
    a.ak = ak;
    a.av = av;
    a.face = face;
    a.o = o;
    a.B = d->batch;
    a.n = n_tok;
    a.H = d->heads;
    a.M = d->streams;
    a.La = int32_t(La);
    a.T = d->tokens_per_frame;
    a.A = d->audio_per_frame;
    a.first_frame = first_frame;
    a.half_window = d->half_window;
    a.n_frames = int32_t(n_frames);
    a.parts = int32_t(parts);
    a.max_keys_pad = int32_t(keys_pad);
    a.o_f32 = o_f32 ? 1 : 0;
    const float scale = d->softmax_scale > 0.f ? d->softmax_scale : 1.f / std::sqrt(float(d->head_dim));
    a.scale_log2 = float(double(scale) * 1.4426950408889634);
    const hipError_t e = tmk::launch_audio_attn_bf16(a, d->head_dim, stream);
    if (e != hipSuccess) return fail(TM_E_DEVICE, "audio attention launch: %s", hipGetErrorString(e));
    return TM_OK;
}

}  // namespace

extern "C" {

tm_status tm_audio_cross_attn_fwd(const tm_audio_desc* d, const void* q, int32_t first_frame,
                                  int32_t n_tok, const void* ak, const void* av,
                                  const int32_t* face, void* o, hipStream_t stream) {
    return audio_fwd(d, q, first_frame, n_tok, ak, av, face, o, false, stream);
}

tm_status tm_audio_cross_attn_fwd_f32out(const tm_audio_desc* d, const void* q,
                                         int32_t first_frame, int32_t n_tok, const void* ak,
                                         const void* av, const int32_t* face, float* o,
                                         hipStream_t stream) {
    return audio_fwd(d, q, first_frame, n_tok, ak, av, face, o, true, stream);
}

const char* tm_last_error(void) { return g_err.c_str(); }

}  // extern "C"
