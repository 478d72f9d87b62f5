// Backward pass of the sparse causal attention, for gfx950 (bf16 MFMA).
//
// The student is trained through the attention of TalkingMachines Sec. 4.2,
// O = softmax(scale * Q K^T) V over each query's allowed key set
// {c_0, c_{a-W}, ..., c_a}. Given dO, the chain rule over the masked row
// softmax gives, with P recomputed from the forward's log-sum-exp:
//
//   delta_i = rowsum(dO_i * O_i)          (= rowsum(P_i * dP_i))
//   dP = dO V^T,  dS = P * (dP - delta)
//   dV = P^T dO,  dQ = scale dS K,  dK = scale dS^T Q
//
// Three kernels, all on the whole-sequence layout [B, L, H, D]:
// - bwd_delta_kernel: delta [B, H, L] in fp32;
// - bwd_dq_kernel: one workgroup of 4 waves per 128-row query tile (tiles
//   never straddle a chunk, so a tile's rows share their key ranges); per
//   64-key tile staged in LDS it recomputes S^T = K Q^T and dP^T = V dO^T and
//   accumulates dQ^T += K^T dS^T, the same operand layouts as the forward's
//   O^T += V^T P^T with row-major V (K^T read with transposing LDS reads);
// - bwd_dkdv_kernel: one workgroup of 8 waves per 256-key tile (32 keys per
//   wave) of one chunk; the queries that see a key chunk c form one range
//   (all of them for c_0, chunks c .. c+W otherwise); per 32-query tile staged
//   in LDS it computes S = Q K^T and dP = dO V^T (one key per lane, queries in
//   registers) and accumulates dV^T += dO^T P and dK^T += Q^T dS, with dO^T and
//   Q^T read with transposing LDS reads. The c_0 tiles, which see every query,
//   are dispatched first.
// P and dS are rounded to bf16 for the MFMAs; accumulation is fp32; results
// are rounded to bf16 once. No atomics: the result is deterministic.

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "tm_device.h"
#include "tm_internal.h"

namespace tmk {
namespace {

constexpr int kDqThreads = 256;    // 4 waves: 128 query rows
constexpr int kDkdvThreads = 512;  // 8 waves: 256 keys

typedef __attribute__((address_space(3))) bf16x8_t lds_bf16x8_t;
typedef __attribute__((address_space(3))) bf16x4_t lds_bf16x4_t;
typedef __attribute__((address_space(3))) unsigned char lds_u8;
typedef __attribute__((address_space(3))) float lds_f32;
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) u32x4_t lds_u32x4_t;

// Per-lane LDS byte offsets inside a row-major tile of D bf16 per row whose
// 16-byte chunks are swizzled by lds_swizzle (rows at multiples of 16 keep
// the pattern):
// - row operand (A of S^T = K Q^T, or A of S = Q K^T): row l32, chunk
//   2*kk + hw, for k-step kk;
// - transposed operand (A of O^T += X^T P^T over 16 rows per step): two
//   transposing reads of rows 4*hw + gi/4 and + 8, element columns
//   32*d + 16*(grp & 1) + 4*(gi & 3); with these the MFMA's k index e of a
//   lane runs over rows 4*hw + e%4 + 8*(e/4), matching the natural output
//   layout of the first product (register i of a lane: row 8*(i/4) + 4*hw + i%4).
template <int D>
struct TileOffsets {
    static constexpr int ROWB = D * 2;
    static constexpr int KK = D / 16;
    static constexpr int DB = D / 32;
    uint32_t row[KK];
    uint32_t tr[2 * DB];
    __device__ __forceinline__ TileOffsets(int lane) {
        const int l32 = lane & 31, hw = lane >> 5;
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) row[kk] = l32 * ROWB + (((2 * kk + hw) ^ lds_swizzle<D>(l32)) << 4);
        const int grp = lane >> 4, gi = lane & 15;
        const int r = 4 * hw + (gi >> 2);
        const int cbase = 2 * (grp & 1) + ((gi & 3) >> 1);
        const int half = (gi & 1) * 8;
#pragma unroll
        for (int d = 0; d < DB; ++d) {
            const int cc = 4 * d + cbase;
            tr[2 * d] = r * ROWB + ((cc ^ lds_swizzle<D>(r)) << 4) + half;
            tr[2 * d + 1] = (r + 8) * ROWB + ((cc ^ lds_swizzle<D>(r + 8)) << 4) + half;
        }
    }
};

template <int D>
__device__ __forceinline__ bf16x8_t read_tr(const lds_u8* tile, uint32_t lo, uint32_t hi) {
    const bf16x4_t a = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)(tile + lo));
    const bf16x4_t b = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)(tile + hi));
    return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}

// Copy `rows` rows (token stride st elements) starting at global row r0 into
// a swizzled LDS tile of n_rows rows; rows at or past r_end repeat row
// r_end - 1 (finite values; callers mask them).
template <int D, int NT>
__device__ __forceinline__ void stage_rows(lds_u8* tile, const __bf16* src, int64_t st, int r0,
                                           int r_end, int n_rows, int tid) {
    constexpr int CPR = D / 8;
    for (int i = tid; i < n_rows * CPR; i += NT) {
        const int r = i / CPR, ch = i % CPR;
        const int gr = min(r0 + r, r_end - 1);
        const u32x4_t x = *reinterpret_cast<const u32x4_t*>(src + gr * st + ch * 8);
        *(lds_u32x4_t*)(tile + r * (D * 2) + ((ch ^ lds_swizzle<D>(r)) << 4)) = x;
    }
}

// ---------------------------------------------------------------------------
// delta = rowsum(dO * O): one thread per (batch, token, head) row
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void bwd_delta_kernel(const __bf16* __restrict__ o,
                                                        const __bf16* __restrict__ dout,
                                                        float* __restrict__ delta, int B, int L,
                                                        int H) {
    const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (idx >= static_cast<int64_t>(B) * L * H) return;
    const int h = static_cast<int>(idx % H);
    const int64_t bi = idx / H;  // b * L + i
    const __bf16* op = o + idx * D;
    const __bf16* dp = dout + idx * D;
    float acc = 0.f;
#pragma unroll
    for (int c = 0; c < D / 8; ++c) {
        const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(op + c * 8);
        const bf16x8_t g = *reinterpret_cast<const bf16x8_t*>(dp + c * 8);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc = fmaf(static_cast<float>(a[e]), static_cast<float>(g[e]), acc);
    }
    const int64_t b = bi / L, i = bi % L;
    delta[(b * H + h) * L + i] = acc;
}

// Key ranges of query chunk a: c_0, and chunks max(1, a - W) .. a, merged.
struct Ranges {
    int n;
    int b0, e0, b1, e1;
};
__device__ __forceinline__ Ranges key_ranges(const BwdArgs& a, int chunk) {
    Ranges r;
    const int ref_end = min(a.ref_tok, a.L);
    if (chunk == 0) {
        r.n = 1;
        r.b0 = 0;
        r.e0 = ref_end;
        return r;
    }
    const int lo_chunk = max(1, chunk - a.window);
    const int b1 = a.ref_tok + (lo_chunk - 1) * a.chunk_tok;
    const int e1 = min(a.ref_tok + chunk * a.chunk_tok, a.L);
    if (b1 <= ref_end) {
        r.n = 1;
        r.b0 = 0;
        r.e0 = e1;
    } else {
        r.n = 2;
        r.b0 = 0;
        r.e0 = ref_end;
        r.b1 = b1;
        r.e1 = e1;
    }
    return r;
}

// Chunk of tile t of a chunk-aligned tiling (ref_tiles tiles for c_0, then
// chunk_tiles per chunk), its first row and its row end.
__device__ __forceinline__ void tile_rows(const BwdArgs& a, int t, int BM, int ref_tiles, int chunk_tiles,
                                          int& chunk, int& r0, int& r1) {
    if (t < ref_tiles) {
        chunk = 0;
        r0 = t * BM;
        r1 = min(r0 + BM, min(a.ref_tok, a.L));
    } else {
        chunk = 1 + (t - ref_tiles) / chunk_tiles;
        const int j = (t - ref_tiles) % chunk_tiles;
        const int cs = a.ref_tok + (chunk - 1) * a.chunk_tok;
        r0 = cs + j * BM;
        r1 = min(min(r0 + BM, cs + a.chunk_tok), a.L);
    }
}

// ---------------------------------------------------------------------------
// dQ: per 128-row query tile, over its key ranges in 64-key tiles
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(kDqThreads) void bwd_dq_kernel(const BwdArgs a) {
    constexpr int ROWB = D * 2, KK = D / 16, DB = D / 32;
    constexpr int BM = kBwdQTile, BN = 64;
    __shared__ __attribute__((aligned(1024))) unsigned char smem[2 * BN * ROWB];
    lds_u8* const Ks = (lds_u8*)smem;
    lds_u8* const Vs = Ks + BN * ROWB;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l32 = lane & 31, hw = lane >> 5;
    const int total = a.q_tiles * a.B * a.H;
    const int id = xcd_logical_id(blockIdx.x, total);
    const int t = id % a.q_tiles;
    const int bh = id / a.q_tiles;
    const int h = bh % a.H, b = bh / a.H;
    int chunk, q0, q1;
    tile_rows(a, t, BM, a.q_ref_tiles, a.q_chunk_tiles, chunk, q0, q1);
    if (q0 >= q1) return;  // a tile past the end of a short last chunk

    const int64_t st = static_cast<int64_t>(a.H) * D;
    const int64_t base = static_cast<int64_t>(b) * a.L * st + h * D;
    const __bf16* qg = static_cast<const __bf16*>(a.q) + base;
    const __bf16* kg = static_cast<const __bf16*>(a.k) + base;
    const __bf16* vg = static_cast<const __bf16*>(a.v) + base;
    const __bf16* dog = static_cast<const __bf16*>(a.dout) + base;
    const float* lse = a.lse + (static_cast<int64_t>(b) * a.H + h) * a.L;
    const float* dl = a.delta + (static_cast<int64_t>(b) * a.H + h) * a.L;

    // this wave's 32 query rows: Q and dO as the B operands of S^T and dP^T
    const int qrow = q0 + wave * 32 + l32;
    const bool row_ok = qrow < q1;
    const int qr = min(qrow, q1 - 1);
    bf16x8_t qf[KK], dof[KK];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
        qf[kk] = *reinterpret_cast<const bf16x8_t*>(qg + qr * st + kk * 16 + hw * 8);
        dof[kk] = *reinterpret_cast<const bf16x8_t*>(dog + qr * st + kk * 16 + hw * 8);
    }
    const float lse2 = lse[qr] * 1.4426950408889634f;
    const float dlt = dl[qr];
    const float c = a.scale_log2;

    const TileOffsets<D> off(lane);
    f32x16_t acc[DB];
#pragma unroll
    for (int d = 0; d < DB; ++d) acc[d] = f32x16_t{};

    const Ranges rg = key_ranges(a, chunk);
    for (int ri = 0; ri < rg.n; ++ri) {
        const int kb0 = ri == 0 ? rg.b0 : rg.b1;
        const int ke = ri == 0 ? rg.e0 : rg.e1;
        for (int k0 = kb0; k0 < ke; k0 += BN) {
            __syncthreads();  // the previous tile is no longer read
            stage_rows<D, kDqThreads>(Ks, kg, st, k0, ke, BN, tid);
            stage_rows<D, kDqThreads>(Vs, vg, st, k0, ke, BN, tid);
            __syncthreads();
            bf16x8_t pf[4];  // dS^T as the B operand, k-step j = 16 keys
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                f32x16_t s = f32x16_t{}, dp = f32x16_t{};
#pragma unroll
                for (int kk = 0; kk < KK; ++kk) {
                    const bf16x8_t kf = *(lds_bf16x8_t*)(Ks + kb * 32 * ROWB + off.row[kk]);
                    const bf16x8_t vf = *(lds_bf16x8_t*)(Vs + kb * 32 * ROWB + off.row[kk]);
                    s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[kk], s, 0, 0, 0);
                    dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, dof[kk], dp, 0, 0, 0);
                }
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int key = k0 + 32 * kb + 8 * (i / 4) + 4 * hw + (i % 4);
                    const float p = key < ke ? __builtin_amdgcn_exp2f(fmaf(s[i], c, -lse2)) : 0.f;
                    const float ds = p * (dp[i] - dlt);
                    pf[2 * kb + i / 8][i % 8] = static_cast<__bf16>(ds);
                }
            }
            // dQ^T += K^T dS^T
#pragma unroll
            for (int j = 0; j < 4; ++j) {
#pragma unroll
                for (int d = 0; d < DB; ++d) {
                    const bf16x8_t kt = read_tr<D>(Ks + 16 * j * ROWB, off.tr[2 * d], off.tr[2 * d + 1]);
                    acc[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kt, pf[j], acc[d], 0, 0, 0);
                }
            }
        }
    }
    if (row_ok) {
        __bf16* dq = static_cast<__bf16*>(a.dq) + base + qrow * st;
        const float sc = a.scale;
#pragma unroll
        for (int d = 0; d < DB; ++d) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                bf16x4_t w;
#pragma unroll
                for (int e = 0; e < 4; ++e) w[e] = static_cast<__bf16>(acc[d][4 * g + e] * sc);
                *reinterpret_cast<bf16x4_t*>(dq + 32 * d + 8 * g + 4 * hw) = w;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// dK, dV: per 128-key tile of one chunk, over the queries that see the chunk
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(kDkdvThreads) void bwd_dkdv_kernel(const BwdArgs a) {
    constexpr int ROWB = D * 2, KK = D / 16, DB = D / 32;
    constexpr int BK = kBwdKTile, BQ = 32;
    __shared__ __attribute__((aligned(1024))) unsigned char smem[2 * BK * ROWB + 2 * BQ * ROWB + 2 * BQ * 4];
    lds_u8* const Ks = (lds_u8*)smem;
    lds_u8* const Vs = Ks + BK * ROWB;
    lds_u8* const Qs = Vs + BK * ROWB;
    lds_u8* const Ds = Qs + BQ * ROWB;  // dO tile
    lds_f32* const lse_s = (lds_f32*)(Ds + BQ * ROWB);
    lds_f32* const dl_s = lse_s + BQ;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l32 = lane & 31, hw = lane >> 5;
    // c_0's key tiles (every query sees them) of all heads first
    const int BH = a.B * a.H;
    const int total = a.k_tiles * BH;
    const int id = xcd_logical_id(blockIdx.x, total);
    int bh, t;
    if (id < a.k_ref_tiles * BH) {
        bh = id / a.k_ref_tiles;
        t = id % a.k_ref_tiles;
    } else {
        const int rest = a.k_tiles - a.k_ref_tiles;
        bh = (id - a.k_ref_tiles * BH) / rest;
        t = a.k_ref_tiles + (id - a.k_ref_tiles * BH) % rest;
    }
    const int h = bh % a.H, b = bh / a.H;
    int chunk, k0, k1;
    tile_rows(a, t, BK, a.k_ref_tiles, a.k_chunk_tiles, chunk, k0, k1);
    if (k0 >= k1) return;
    // queries that see key chunk `chunk`
    int qa, qb;
    if (chunk == 0) {
        qa = 0;
        qb = a.L;
    } else {
        qa = a.ref_tok + (chunk - 1) * a.chunk_tok;
        qb = min(a.ref_tok + (chunk + a.window) * a.chunk_tok, a.L);
    }

    const int64_t st = static_cast<int64_t>(a.H) * D;
    const int64_t base = static_cast<int64_t>(b) * a.L * st + h * D;
    const __bf16* qg = static_cast<const __bf16*>(a.q) + base;
    const __bf16* kg = static_cast<const __bf16*>(a.k) + base;
    const __bf16* vg = static_cast<const __bf16*>(a.v) + base;
    const __bf16* dog = static_cast<const __bf16*>(a.dout) + base;
    const float* lse = a.lse + (static_cast<int64_t>(b) * a.H + h) * a.L;
    const float* dl = a.delta + (static_cast<int64_t>(b) * a.H + h) * a.L;

    stage_rows<D, kDkdvThreads>(Ks, kg, st, k0, k1, BK, tid);
    stage_rows<D, kDkdvThreads>(Vs, vg, st, k0, k1, BK, tid);

    const TileOffsets<D> off(lane);
    // this wave's 32 keys as the B operands of S = Q K^T and dP = dO V^T
    const uint32_t krow = (wave * 32 + l32) * ROWB;
    const int kswz = lds_swizzle<D>(l32);  // (wave * 32 + l32) % 16 == l32 % 16
    f32x16_t dk[DB], dv[DB];
#pragma unroll
    for (int d = 0; d < DB; ++d) dk[d] = dv[d] = f32x16_t{};
    const float c = a.scale_log2;

    for (int q0 = qa; q0 < qb; q0 += BQ) {
        __syncthreads();  // the previous query tile is no longer read (and K/V are staged)
        stage_rows<D, kDkdvThreads>(Qs, qg, st, q0, qb, BQ, tid);
        stage_rows<D, kDkdvThreads>(Ds, dog, st, q0, qb, BQ, tid);
        if (tid < BQ) {
            const int qr = min(q0 + tid, qb - 1);
            lse_s[tid] = lse[qr] * 1.4426950408889634f;
            dl_s[tid] = dl[qr];
        }
        __syncthreads();
        f32x16_t s = f32x16_t{}, dp = f32x16_t{};
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
            const bf16x8_t qa_f = *(lds_bf16x8_t*)(Qs + off.row[kk]);
            const bf16x8_t da_f = *(lds_bf16x8_t*)(Ds + off.row[kk]);
            const int pos = ((2 * kk + hw) ^ kswz) << 4;
            const bf16x8_t kb_f = *(lds_bf16x8_t*)(Ks + krow + pos);
            const bf16x8_t vb_f = *(lds_bf16x8_t*)(Vs + krow + pos);
            s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa_f, kb_f, s, 0, 0, 0);
            dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(da_f, vb_f, dp, 0, 0, 0);
        }
        // register i: query 8*(i/4) + 4*hw + i%4 of the tile, key l32 of the wave
        bf16x8_t pf[2], sf[2];
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int qi = 8 * (i / 4) + 4 * hw + (i % 4);
            const float p = q0 + qi < qb ? __builtin_amdgcn_exp2f(fmaf(s[i], c, -lse_s[qi])) : 0.f;
            pf[i / 8][i % 8] = static_cast<__bf16>(p);
            sf[i / 8][i % 8] = static_cast<__bf16>(p * (dp[i] - dl_s[qi]));
        }
        // dV^T += dO^T P and dK^T += Q^T dS, over the tile's 32 queries (2 k-steps)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
#pragma unroll
            for (int d = 0; d < DB; ++d) {
                const bf16x8_t dt = read_tr<D>(Ds + 16 * j * ROWB, off.tr[2 * d], off.tr[2 * d + 1]);
                const bf16x8_t qt = read_tr<D>(Qs + 16 * j * ROWB, off.tr[2 * d], off.tr[2 * d + 1]);
                dv[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(dt, pf[j], dv[d], 0, 0, 0);
                dk[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qt, sf[j], dk[d], 0, 0, 0);
            }
        }
    }
    const int key = k0 + wave * 32 + l32;
    if (key < k1) {
        __bf16* dkp = static_cast<__bf16*>(a.dk) + base + key * st;
        __bf16* dvp = static_cast<__bf16*>(a.dv) + base + key * st;
        const float sc = a.scale;
#pragma unroll
        for (int d = 0; d < DB; ++d) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                bf16x4_t wk, wv;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    wk[e] = static_cast<__bf16>(dk[d][4 * g + e] * sc);
                    wv[e] = static_cast<__bf16>(dv[d][4 * g + e]);
                }
                *reinterpret_cast<bf16x4_t*>(dkp + 32 * d + 8 * g + 4 * hw) = wk;
                *reinterpret_cast<bf16x4_t*>(dvp + 32 * d + 8 * g + 4 * hw) = wv;
            }
        }
    }
}

template <int D>
hipError_t launch_bwd(const BwdArgs& a, hipStream_t s) {
    const int64_t rows = static_cast<int64_t>(a.B) * a.L * a.H;
    const int64_t g0 = (rows + 255) / 256;
    const int64_t g1 = static_cast<int64_t>(a.q_tiles) * a.B * a.H;
    const int64_t g2 = static_cast<int64_t>(a.k_tiles) * a.B * a.H;
    if (g0 > INT32_MAX || g1 > INT32_MAX || g2 > INT32_MAX) return hipErrorInvalidValue;
    hipLaunchKernelGGL(bwd_delta_kernel<D>, dim3(static_cast<unsigned>(g0)), dim3(256), 0, s,
                       static_cast<const __bf16*>(a.o), static_cast<const __bf16*>(a.dout), a.delta,
                       a.B, a.L, a.H);
    hipLaunchKernelGGL(bwd_dq_kernel<D>, dim3(static_cast<unsigned>(g1)), dim3(kDqThreads), 0, s, a);
    hipLaunchKernelGGL(bwd_dkdv_kernel<D>, dim3(static_cast<unsigned>(g2)), dim3(kDkdvThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_bwd_bf16(const BwdArgs& a, int head_dim, hipStream_t s) {
    if (head_dim == 128) return launch_bwd<128>(a, s);
    if (head_dim == 64) return launch_bwd<64>(a, s);
    return hipErrorInvalidValue;
}

}  // namespace tmk
