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
//   64-key tile, loaded straight into LDS while the previous tile computes,
//   it recomputes S^T = K Q^T and dP^T = V dO^T and accumulates
//   dQ^T += K^T dS^T, the same operand layouts as the forward's
//   O^T += V^T P^T with row-major V (K^T read with transposing LDS reads);
// - bwd_dkdv_kernel: one workgroup of 4 waves per 128-key tile of one chunk
//   (two workgroups share a CU, so each SIMD runs two independent waves);
//   the queries that see a key chunk c form one range (all of them for c_0,
//   chunks c .. c+W otherwise); per 32-query stage, loaded straight into LDS
//   while the previous stage computes, it forms S = Q K^T and dP = dO V^T
//   (one key per lane) and accumulates dV^T += dO^T P and dK^T += Q^T dS,
//   with dO^T and Q^T read with transposing LDS reads. The c_0 tiles, which
//   see every query, are dispatched first.
// P and dS are rounded to bf16 for the MFMAs; accumulation is fp32; results
// are rounded to bf16 once. No atomics: the result is deterministic.

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <atomic>
#include <type_traits>

#include "tm_device.h"
#include "tm_internal.h"

namespace tmk {
namespace {

constexpr int kDqThreads = 256;    // 4 waves: 128 query rows; two workgroups per CU
constexpr int kDkdvThreads = 256;  // 4 waves: 128 keys; two workgroups per CU

typedef __attribute__((address_space(3))) bf16x8_t lds_bf16x8_t;
typedef __attribute__((address_space(3))) bf16x4_t lds_bf16x4_t;
typedef __attribute__((address_space(3))) unsigned char lds_u8;
typedef __attribute__((address_space(3))) float lds_f32;
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) f32x4_t lds_f32x4_t;

// LDS tiles of both gradient kernels (K and V in dQ; Q, dO and V in dK/dV)
// put 16-byte chunk c of row `row` at c ^ tr_swizzle<D>(row).
// Per-lane LDS byte offsets inside such a tile (rows at multiples of 16 keep
// the pattern):
// - row operand (A of S^T = K Q^T, or A of S = Q K^T): row l32, chunk
//   2*kk + hw, for k-step kk: row(kk);
// - transposed operand (A of X^T-times-P products over 16 rows per step):
//   two transposing reads, tr_lo(d) and tr_hi(d), of rows 4*hw + gi/4 and
//   + 8 at element columns 32*d + 16*(grp & 1) + 4*(gi & 3); with these the
//   MFMA's k index e of a lane runs over rows 4*hw + e%4 + 8*(e/4), matching
//   the natural output layout of the first product (register i of a lane:
//   row 8*(i/4) + 4*hw + i%4).
// The chunk is 2*kk + hw or 4*d + cbase, and the swizzle's XOR only touches
// the chunk bits, so row(kk) = row0 ^ (kk << 5) and tr_lo(d) = tr0 ^ (d << 6):
// three registers instead of sixteen. pinned() makes a stage derive them anew
// (one XOR per use) rather than have the compiler keep all of them.
template <int D>
struct TileBases {
    static constexpr int ROWB = D * 2;
    uint32_t row0, tr0, tr8;
    __device__ __forceinline__ TileBases(int lane) {
        const int l32 = lane & 31, hw = lane >> 5;
        row0 = l32 * ROWB + ((hw ^ tr_swizzle<D>(l32)) << 4);
        const int grp = lane >> 4, gi = lane & 15;
        const int r = 4 * hw + (gi >> 2);
        const int cbase = 2 * (grp & 1) + ((gi & 3) >> 1);
        const int half = (gi & 1) * 8;
        tr0 = r * ROWB + ((cbase ^ tr_swizzle<D>(r)) << 4) + half;
        tr8 = r * ROWB + ((cbase ^ tr_swizzle<D>(r + 8)) << 4) + half;
    }
    __device__ __forceinline__ TileBases pinned() const {
        TileBases t = *this;
        asm volatile("" : "+v"(t.row0), "+v"(t.tr0), "+v"(t.tr8));
        return t;
    }
    __device__ __forceinline__ uint32_t row(int kk) const { return row0 ^ (kk << 5); }
    __device__ __forceinline__ uint32_t tr_lo(int d) const { return tr0 ^ (d << 6); }
    __device__ __forceinline__ uint32_t tr_hi(int d) const { return (tr8 ^ (d << 6)) + 8 * ROWB; }
};

template <int D>
__device__ __forceinline__ bf16x8_t read_tr(const lds_u8* tile, uint32_t lo, uint32_t hi) {
    const bf16x4_t a = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)(tile + lo));
    const bf16x4_t b = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)(tile + hi));
    return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
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
// Each wave owns 32 query rows and holds their Q and dO fragments (the B
// operands of S^T = K Q^T and dP^T = V dO^T) and their dQ^T accumulators in
// registers. The key tiles of the tile's (at most two) key ranges form one
// sequence; each tile's K and V rows arrive by direct global->LDS loads into
// two alternating buffers, the next tile's loads in flight during the current
// tile's arithmetic; one barrier per tile.
template <int D>
__global__ __launch_bounds__(kDqThreads, 2) void bwd_dq_kernel(const BwdArgs a) {
    constexpr int ROWB = D * 2, KK = D / 16, DB = D / 32, CPR = D / 8;
    constexpr int BM = kBwdQTile, BN = 64;
    constexpr int NW = kDqThreads / 64;         // waves
    constexpr int KT = BN * ROWB;               // one tensor's key tile in LDS
    constexpr int BUF = 2 * KT;                 // K tile, then V tile
    constexpr int NBW = KT / 1024 / NW;         // 1-KB direct loads per wave, tensor and tile
    static_assert(NBW >= 1 && NBW * NW * 1024 == KT, "key tile must split over the waves");
    static_assert(BM == NW * 32, "32 query rows per wave");
    __shared__ __attribute__((aligned(1024))) unsigned char smem[2 * BUF];
    lds_u8* const L = (lds_u8*)smem;
    const uint32_t lds_base = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(L));

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l32 = lane & 31, hw = lane >> 5;
    // The chunks' query tiles (which see c_0 and W + 1 chunks of keys) first,
    // grouped per XCD so that a head's tiles share an L2; c_0's tiles (which
    // see c_0 only) last, in plain dispatch order, so that they spread over
    // the XCDs and fill the end of the grid.
    const int BH = a.B * a.H;
    const int rest = a.q_tiles - a.q_ref_tiles;
    const int n_chunk = rest * BH;
    int bh, t;
    if (static_cast<int>(blockIdx.x) < n_chunk) {
        const int id = xcd_logical_id(blockIdx.x, n_chunk);
        bh = id / rest;
        t = a.q_ref_tiles + id % rest;
    } else {
        const int r = blockIdx.x - n_chunk;
        bh = r / a.q_ref_tiles;
        t = r % a.q_ref_tiles;
    }
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
    // the Q/dO loads land before any direct load is issued
    wait_lds_dma();

    // key tile j of the sequence: first key k0 and end ke of its range
    const Ranges rg = key_ranges(a, chunk);
    const int n0 = (rg.e0 - rg.b0 + BN - 1) / BN;
    const int nt = n0 + (rg.n == 2 ? (rg.e1 - rg.b1 + BN - 1) / BN : 0);
    auto tile_at = [&](int j, int& k0, int& ke) __attribute__((always_inline)) {
        if (j < n0) {
            k0 = rg.b0 + j * BN;
            ke = rg.e0;
        } else {
            k0 = rg.b1 + (j - n0) * BN;
            ke = rg.e1;
        }
    };
    // Direct loads of key tile j into buffer u (rows past ke repeat row
    // ke - 1: finite values, masked below), swizzled as in the dK/dV kernel.
    auto issue = [&](int j, int u) __attribute__((always_inline)) {
        int k0, ke;
        tile_at(j, k0, ke);
        const int last = ke - 1 - k0;
        const void* ks = uniform_ptr(kg + k0 * st);
        const void* vs = uniform_ptr(vg + k0 * st);
#pragma unroll
        for (int i = 0; i < NBW; ++i) {
            const int blk = i * NW + wave;
            const int ch = blk * 64 + lane;
            const int row = ch / CPR;
            const int gc = (ch % CPR) ^ tr_swizzle<D>(row);
            const uint32_t voff = static_cast<uint32_t>((min(row, last) * st + gc * 8) * 2);
            const uint32_t l = lds_base + u * BUF + blk * 1024;
            lds_dma16x2(ks, voff, l, vs, voff, l + KT);
        }
    };

    const TileBases<D> tb(lane);
    f32x16_t acc[DB];
#pragma unroll
    for (int d = 0; d < DB; ++d) acc[d] = f32x16_t{};

    // Key tile j from buffer U: S^T = K Q^T and dP^T = V dO^T per 32-key
    // block kb (register i: key 32*kb + 8*(i/4) + 4*hw + i%4, query l32),
    // dS^T as the B operand of dQ^T += K^T dS^T (k-step = 16 keys). Only a
    // range's last tile can hold keys past the range (MASKED).
    auto tile = [&](auto ucst, auto maskc, int k0, int ke) __attribute__((always_inline)) {
        constexpr int U = decltype(ucst)::value;
        constexpr bool MASKED = decltype(maskc)::value;
        const lds_u8* Ks = L + U * BUF;
        const lds_u8* Vs = Ks + KT;
        const TileBases<D> off = tb.pinned();
        bf16x8_t pf[4];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            f32x16_t s = f32x16_t{}, dp = f32x16_t{};
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) {
                const bf16x8_t kf = *(const lds_bf16x8_t*)(Ks + kb * 32 * ROWB + off.row(kk));
                const bf16x8_t vf = *(const lds_bf16x8_t*)(Vs + kb * 32 * ROWB + off.row(kk));
                s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[kk], s, 0, 0, 0);
                dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, dof[kk], dp, 0, 0, 0);
            }
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                float p = __builtin_amdgcn_exp2f(fmaf(s[i], c, -lse2));
                if constexpr (MASKED) p = k0 + 32 * kb + 8 * (i / 4) + 4 * hw + (i % 4) < ke ? p : 0.f;
                pf[2 * kb + i / 8][i % 8] = static_cast<__bf16>(p * (dp[i] - dlt));
            }
        }
#pragma unroll
        for (int j4 = 0; j4 < 4; ++j4) {
#pragma unroll
            for (int d = 0; d < DB; ++d) {
                const bf16x8_t kt = read_tr<D>(Ks + 16 * j4 * ROWB, off.tr_lo(d), off.tr_hi(d));
                acc[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kt, pf[j4], acc[d], 0, 0, 0);
            }
        }
    };
    auto compute = [&](auto ucst, int j) __attribute__((always_inline)) {
        int k0, ke;
        tile_at(j, k0, ke);
        if (ke - k0 >= BN) {
            tile(ucst, std::false_type{}, k0, ke);
        } else {
            tile(ucst, std::true_type{}, k0, ke);
        }
    };

    issue(0, 0);
    wait_lds_dma();
    __syncthreads();
    for (int j = 0; j < nt; j += 2) {
        // buffer 1 was last read in the previous tile, before the barrier
        if (j + 1 < nt) issue(j + 1, 1);
        compute(std::integral_constant<int, 0>{}, j);
        wait_lds_dma();
        __syncthreads();
        if (j + 1 >= nt) break;
        if (j + 2 < nt) issue(j + 2, 0);
        compute(std::integral_constant<int, 1>{}, j + 1);
        wait_lds_dma();
        __syncthreads();
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
// Each wave owns 32 keys and holds their K fragments (the B operand of
// S = Q K^T) and their dK^T and dV^T accumulators in registers (about 240 per
// lane, so two waves fit on a SIMD); the workgroup's V rows (the B operand of
// dP = dO V^T) sit in LDS. The 32-query stages of Q, dO, lse and delta arrive
// by direct global->LDS loads into two alternating buffers, the next stage's
// loads in flight during the current stage's arithmetic; one barrier per
// stage. Two workgroups per CU keep the SIMDs' two waves out of step, so that
// one wave's softmax arithmetic can overlap the other's MFMAs (partly: two
// waves that both alternate the two kinds of work overlap only in part).
template <int D>
__global__ __launch_bounds__(kDkdvThreads, 2) void bwd_dkdv_kernel(const BwdArgs a) {
    constexpr int ROWB = D * 2, KK = D / 16, DB = D / 32, CPR = D / 8;
    constexpr int BQ = 32;                      // queries per stage
    constexpr int NW = kDkdvThreads / 64;       // waves
    constexpr int TILE = BQ * ROWB;             // one tensor's stage tile in LDS
    constexpr int STAGE = 2 * TILE;             // Q tile, then dO tile
    constexpr int NB = TILE / 1024;             // 1-KB direct loads per tensor and stage
    static_assert(NB % NW == 0, "stage tile must split over the waves");
    constexpr int VEC = 2 * STAGE;              // lse and delta: 2 buffers x 64 floats each
    constexpr int VT = VEC + 4 * 256;           // V rows of the workgroup's keys
    static_assert(kBwdKTile == NW * 32, "32 keys per wave");
    __shared__ __attribute__((aligned(1024))) unsigned char smem[VT + kBwdKTile * ROWB];
    lds_u8* const L = (lds_u8*)smem;
    const uint32_t lds_base = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(L));

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l32 = lane & 31, hw = lane >> 5;
    // c_0's key tiles (every query sees them: 3.5x the work of a chunk's
    // tile at W = 1) of all heads first, in plain dispatch order so that they
    // spread over the 8 XCDs (grouping them per XCD would leave one XCD with
    // all of them); the chunks' tiles after them, grouped per XCD so that a
    // head's tiles share an L2.
    const int BH = a.B * a.H;
    const int n_ref = a.k_ref_tiles * BH;
    int bh, t;
    if (static_cast<int>(blockIdx.x) < n_ref) {
        bh = blockIdx.x / a.k_ref_tiles;
        t = blockIdx.x % a.k_ref_tiles;
    } else {
        const int rest = a.k_tiles - a.k_ref_tiles;
        const int id = xcd_logical_id(blockIdx.x - n_ref, rest * BH);
        bh = id / rest;
        t = a.k_ref_tiles + id % rest;
    }
    const int h = bh % a.H, b = bh / a.H;
    int chunk, k0, k1;
    tile_rows(a, t, kBwdKTile, a.k_ref_tiles, a.k_chunk_tiles, chunk, k0, k1);
    if (k0 >= k1) return;
    // queries [qbeg, qend) see key chunk `chunk`
    int qbeg, qend;
    if (chunk == 0) {
        qbeg = 0;
        qend = a.L;
    } else {
        qbeg = a.ref_tok + (chunk - 1) * a.chunk_tok;
        qend = min(a.ref_tok + (chunk + a.window) * a.chunk_tok, a.L);
    }

    const int64_t st = static_cast<int64_t>(a.H) * D;
    const int64_t base = static_cast<int64_t>(b) * a.L * st + h * D;
    const __bf16* qg = static_cast<const __bf16*>(a.q) + base;
    const __bf16* kg = static_cast<const __bf16*>(a.k) + base;
    const __bf16* vg = static_cast<const __bf16*>(a.v) + base;
    const __bf16* dog = static_cast<const __bf16*>(a.dout) + base;
    const float* lse = a.lse + (static_cast<int64_t>(b) * a.H + h) * a.L;
    const float* dl = a.delta + (static_cast<int64_t>(b) * a.H + h) * a.L;

    // Direct loads of the stage starting at query q0 into buffer u: rows past
    // qend repeat row qend - 1 (finite values; seal() below zeroes their P
    // and dS). Each 1-KB block
    // holds 64 consecutive 16-byte LDS chunks of the swizzled tile; the lane
    // whose chunk is logical chunk gc of row `row` fetches that chunk.
    auto issue = [&](int q0, int u) __attribute__((always_inline)) {
        const int last = qend - 1 - q0;
        const void* qs = uniform_ptr(qg + q0 * st);
        const void* ds = uniform_ptr(dog + q0 * st);
#pragma unroll
        for (int i = 0; i < NB / NW; ++i) {
            const int blk = i * NW + wave;
            const int ch = blk * 64 + lane;
            const int row = ch / CPR;
            const int gc = (ch % CPR) ^ tr_swizzle<D>(row);
            const uint32_t voff = static_cast<uint32_t>((min(row, last) * st + gc * 8) * 2);
            const uint32_t l = lds_base + u * STAGE + blk * 1024;
            lds_dma16x2(qs, voff, l, ds, voff, l + TILE);
        }
        if (wave == NW - 1) {
            const uint32_t vo = static_cast<uint32_t>(min(lane, last) * 4);
            lds_dma4x2(uniform_ptr(lse + q0), vo, lds_base + VEC + u * 256, uniform_ptr(dl + q0), vo,
                       lds_base + VEC + 512 + u * 256);
        }
    };

    // this wave's keys: k0 + 32 * wave + l32
    const int kw = k0 + 32 * wave;
    const bool busy = kw < k1;
    bf16x8_t kf[KK];
    {
        const int kr = min(kw + l32, k1 - 1);
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
            kf[kk] = *reinterpret_cast<const bf16x8_t*>(kg + kr * st + kk * 16 + hw * 8);
    }
    // this wave's 32 V rows into LDS (rows past k1 repeat row k1 - 1)
    {
        const int vk = min(kw, k1 - 1);
        const void* vs = uniform_ptr(vg + static_cast<int64_t>(vk) * st);
        const int vlast = k1 - 1 - vk;
#pragma unroll
        for (int i = 0; i < 32 * ROWB / 1024; i += 2) {
            uint32_t vo[2];
#pragma unroll
            for (int m = 0; m < 2; ++m) {
                const int ch = (i + m) * 64 + lane;
                const int row = ch / CPR;
                const int gc = (ch % CPR) ^ tr_swizzle<D>(row);
                vo[m] = static_cast<uint32_t>((min(row, vlast) * st + gc * 8) * 2);
            }
            const uint32_t l = lds_base + VT + wave * 32 * ROWB + i * 1024;
            lds_dma16x2(vs, vo[0], l, vs, vo[1], l + 1024);
        }
    }
    // the K loads and the V rows land before any stage load is issued
    wait_lds_dma();

    const TileBases<D> tb(lane);
    f32x16_t dk[DB], dv[DB];
#pragma unroll
    for (int d = 0; d < DB; ++d) dk[d] = dv[d] = f32x16_t{};
    const float c = a.scale_log2;

    // One stage from buffer U: S = Q K^T and dP = dO V^T (register i: query
    // 8*(i/4) + 4*hw + i%4 of the stage, key l32 of the wave), then
    // dV^T += dO^T P and dK^T += Q^T dS over the stage's 32 queries.
    auto compute = [&](auto ucst, int q0) __attribute__((always_inline)) {
        constexpr int U = decltype(ucst)::value;
        const lds_u8* Qb = L + U * STAGE;
        const lds_u8* Db = Qb + TILE;
        const lds_u8* Vw = L + VT + wave * 32 * ROWB;
        const lds_f32* ls = (const lds_f32*)(L + VEC + U * 256);
        const lds_f32* dls = (const lds_f32*)(L + VEC + 512 + U * 256);
        const TileBases<D> off = tb.pinned();
        // the two chains interleaved: one's MFMA covers the other's LDS reads;
        // the operands of k-step kk + 2 are read while k-step kk runs
        f32x16_t s = f32x16_t{}, dp = f32x16_t{};
        bf16x8_t qa[3], da[3], vb[3];
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            qa[kk] = *(const lds_bf16x8_t*)(Qb + off.row(kk));
            da[kk] = *(const lds_bf16x8_t*)(Db + off.row(kk));
            vb[kk] = *(const lds_bf16x8_t*)(Vw + off.row(kk));
        }
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
            if (kk + 2 < KK) {
                qa[(kk + 2) % 3] = *(const lds_bf16x8_t*)(Qb + off.row(kk + 2));
                da[(kk + 2) % 3] = *(const lds_bf16x8_t*)(Db + off.row(kk + 2));
                vb[(kk + 2) % 3] = *(const lds_bf16x8_t*)(Vw + off.row(kk + 2));
            }
            s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa[kk % 3], kf[kk], s, 0, 0, 0);
            dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(da[kk % 3], vb[kk % 3], dp, 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
        }
        // P and dS, 4 consecutive queries at a time (their lse, +inf for rows
        // past qend so that P = 0, and delta)
        bf16x8_t pf[2], sf[2];
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
            const int q4 = 8 * g4 + 4 * hw;
            const f32x4_t x = *(const lds_f32x4_t*)(ls + q4);
            const f32x4_t y = *(const lds_f32x4_t*)(dls + q4);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int i = 4 * g4 + e;
                const float ml = x[e] * 1.4426950408889634f;
                const float p = __builtin_amdgcn_exp2f(fmaf(s[i], c, -ml));
                pf[i / 8][i % 8] = static_cast<__bf16>(p);
                sf[i / 8][i % 8] = static_cast<__bf16>(p * (dp[i] - y[e]));
            }
        }
#pragma unroll
        for (int j = 0; j < 2; ++j) {
#pragma unroll
            for (int d = 0; d < DB; ++d) {
                const bf16x8_t dt = read_tr<D>(Db + 16 * j * ROWB, off.tr_lo(d), off.tr_hi(d));
                dv[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(dt, pf[j], dv[d], 0, 0, 0);
                const bf16x8_t qt = read_tr<D>(Qb + 16 * j * ROWB, off.tr_lo(d), off.tr_hi(d));
                dk[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qt, sf[j], dk[d], 0, 0, 0);
            }
        }
    };

    // The last stage can hold rows past qend (their loads repeat row
    // qend - 1): once its loads have landed, their lse becomes +inf, so that
    // their P and dS are exactly zero and no stage needs a per-row mask.
    auto seal = [&](int u, int q0) __attribute__((always_inline)) {
        const int rows = qend - q0;
        if (rows < BQ) {
            if (tid >= rows && tid < BQ) ((lds_f32*)(L + VEC + u * 256))[tid] = __builtin_inff();
            __syncthreads();
        }
    };
    const int n_st = (qend - qbeg + BQ - 1) / BQ;
    issue(qbeg, 0);
    wait_lds_dma();
    __syncthreads();
    for (int ts = 0; ts < n_st; ts += 2) {
        const int q0 = qbeg + ts * BQ;
        if (ts + 1 < n_st) issue(q0 + BQ, 1);
        seal(0, q0);
        if (busy) compute(std::integral_constant<int, 0>{}, q0);
        wait_lds_dma();
        __syncthreads();
        if (ts + 1 >= n_st) break;
        if (ts + 2 < n_st) issue(q0 + 2 * BQ, 0);
        seal(1, q0 + BQ);
        if (busy) compute(std::integral_constant<int, 1>{}, q0 + BQ);
        wait_lds_dma();
        __syncthreads();
    }

    const float sc = a.scale;
    const int key = kw + l32;
    if (key < k1) {
        __bf16* dkp = static_cast<__bf16*>(a.dk) + base + key * st;
        __bf16* dvp = static_cast<__bf16*>(a.dv) + base + key * st;
#pragma unroll
        for (int d = 0; d < DB; ++d) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                bf16x4_t wk, wv;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    wk[e] = static_cast<__bf16>(dk[d][4 * q + e] * sc);
                    wv[e] = static_cast<__bf16>(dv[d][4 * q + e]);
                }
                *reinterpret_cast<bf16x4_t*>(dkp + 32 * d + 8 * q + 4 * hw) = wk;
                *reinterpret_cast<bf16x4_t*>(dvp + 32 * d + 8 * q + 4 * hw) = wv;
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

// Workspace of the allocation-free backward entry point: delta for up to
// kBwdScratchFloats (batch, head, token) rows, in a device-global array that
// every GPU the library runs on holds until the process ends. Host code never
// passes this symbol to a kernel (on the host it names a stand-in, not the
// device copy): it uses the address hipGetSymbolAddress returns for the
// current device.
__device__ __align__(256) float scratch[kBwdScratchFloats];

constexpr int kMaxScratchDevices = 64;

}  // namespace

hipError_t launch_attn_bwd_bf16(const BwdArgs& a, int head_dim, hipStream_t s) {
    if (head_dim == 128) return launch_bwd<128>(a, s);
    if (head_dim == 64) return launch_bwd<64>(a, s);
    return hipErrorInvalidValue;
}

hipError_t bwd_scratch_address(float** out) {
    // One address per device, looked up once, with that device current
    // (every GPU holds its own copy of the array).
    static std::atomic<float*> addr[kMaxScratchDevices];
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxScratchDevices) return hipErrorInvalidDevice;
    float* p = addr[dev].load(std::memory_order_acquire);
    if (p == nullptr) {
        void* q = nullptr;
        e = hipGetSymbolAddress(&q, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (q == nullptr) return hipErrorInvalidSymbol;
        p = static_cast<float*>(q);
        addr[dev].store(p, std::memory_order_release);  // concurrent first calls store the same value
    }
    *out = p;
    return hipSuccess;
}

}  // namespace tmk
