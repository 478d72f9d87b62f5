// Sparse causal attention forward for gfx950 (MI355X, CDNA4).
//
// Computes, for every query row i of chunk a, O_i = softmax_j(scale * q_i.k_j) v_j
// over the keys j of {c_0, c_{a-W}, ..., c_a} (TalkingMachines, Sec. 4.2: the
// sparse attention pattern and its attention equation). The key set of a query
// chunk is a union of at most a few contiguous key ranges; query tiles never
// straddle a chunk, so every row of a tile shares its ranges, key tiles are
// visited only inside those ranges (masked blocks are never loaded), and only
// the last key tile of a range needs a column mask.
//
// bf16 kernel: one workgroup of 8 waves (two per SIMD) per 256-row query tile,
// 32 query rows per wave; all 8 waves share each K/V tile staged in LDS.
// Per 64-key tile the work is
//   S^T (keys x queries) = K Q^T with v_mfma_f32_32x32x16_bf16, K from LDS,
//     Q^T held in registers for the whole loop;
//   the softmax in fp32 on the MFMA output layout (each lane owns one query
//     column and half of its keys): x = S*scale*log2(e) - m against a lazily
//     raised running max m, P = exp2(x), rounded to bf16 for the P V product,
//     row sums of P in fp32;
//   O^T (head_dim x queries) += V^T P^T with the same MFMA, P^T straight from
//     registers. From the KV cache, whose V blocks are stored dimension-major,
//     the V tile lands in LDS as V^T and each operand is one 16-byte read; the
//     K rows are fed to the S MFMA in a permuted order that makes each lane's
//     P^T elements 8 consecutive keys. From row-major V (whole-sequence calls
//     on caller tensors) the operand is read with the gfx950 transposing read.
// The loop is software-pipelined so that every wave keeps the matrix core fed
// with its own VALU work in between (a wave's VALU work overlaps the MFMAs of
// the same wave far better than those of the other wave on its SIMD): while
// the MFMAs of S(t+1) run, the same wave forms P(t); while those of P(t) V(t)
// run, it scales S(t+1). Each MFMA is preceded by the LDS read of the operand
// fragment four MFMAs ahead. K/V tiles stream through four LDS buffers per
// tensor, filled by direct global->LDS loads two (V) and four (K) tiles ahead,
// with one barrier per tile.
//
// fp32 kernel: a plain VALU kernel (4 lanes per query row, exact running max)
// for fp32 inputs; it exists for correctness at small sizes.

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "tm_device.h"
#include "tm_internal.h"

namespace tmk {
namespace {

typedef __attribute__((address_space(3))) bf16x4_t lds_bf16x4_t;
typedef __attribute__((address_space(3))) bf16x8_t lds_bf16x8_t;
typedef __attribute__((address_space(3))) unsigned char lds_u8;

// Threads per workgroup of the bf16 kernel: 8 waves (two per SIMD) sharing
// every K/V tile staged in LDS.
constexpr int kBf16Threads = 512;
// Wait until at most N LDS operations (and scalar loads) of this wave are
// outstanding; vector-memory and export counts are left unconstrained.
template <int N>
__device__ __forceinline__ void wait_lds_reads() {
    static_assert(N >= 0 && N < 16, "lgkmcnt field");
    __builtin_amdgcn_s_waitcnt(0xC07F | (N << 8));
}

// The same, except that the newest N direct loads may still be in flight
// (vector-memory operations complete in issue order for this count).
template <int N>
__device__ __forceinline__ void wait_lds_dma_but() {
    static_assert(N >= 0 && N < 16, "vmcnt field");
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0 | N);
}

// Keeps x in a register at this point of the program: the empty statement
// takes x as input and output, so the computation of x cannot be moved past
// it (the compiler would otherwise sink work that is only used after a branch
// or a barrier, away from the MFMAs it is meant to overlap).
// threadIdx.x, which the compiler cannot fold into an earlier copy.
__device__ __forceinline__ int fresh_thread_index() {
    int v = static_cast<int>(threadIdx.x);
    asm volatile("" : "+v"(v));
    return v;
}

__device__ __forceinline__ float pin(float x) {
    asm volatile("" : "+v"(x));
    return x;
}

// Query rows [q0, q1) of tile `tile` and its key ranges. Mode 0 reads the
// ranges from the kernel arguments; mode 1 derives them from the geometry.
struct TileRanges {
    int q0, q1;
    int n;         // number of ranges
    int b0, e0;    // mode 1 ranges (at most two)
    int b1, e1;
};

// Rows [q0, q1) of tile `idx` among the `nt` tiles that cover the rows
// [begin, end) of one chunk: the chunk's 32-row blocks are split as evenly as
// possible, so every tile gets the same number of blocks give or take one
// (at most BM / 32 since nt >= (end - begin) / BM) and tiles take about equally
// long; only the chunk's last block may be partial.
template <int BM>
__device__ __forceinline__ void split_rows(int begin, int end, int nt, int idx, int& q0, int& q1) {
    const int blocks = (end - begin + 31) / 32;
    q0 = begin + 32 * ((idx * blocks) / nt);
    q1 = min(begin + 32 * (((idx + 1) * blocks) / nt), end);
}

template <int BM>
__device__ __forceinline__ TileRanges plan_tile(const AttnArgs& a, int tile) {
    TileRanges t;
    if (a.mode == 0) {
        split_rows<BM>(0, a.Lq, a.n_qtiles, tile, t.q0, t.q1);
        t.n = a.n_ranges;
        t.b0 = t.e0 = t.b1 = t.e1 = 0;
        return t;
    }
    // Mode 1: tiles are ordered heaviest first (the last chunks see the most
    // keys), so walk the natural order backwards.
    const int nat = a.n_qtiles - 1 - tile;
    int chunk;
    if (nat < a.ref_tiles) {
        chunk = 0;
        split_rows<BM>(0, a.ref_tok, a.ref_tiles, nat, t.q0, t.q1);
    } else {
        const int u = nat - a.ref_tiles;
        chunk = 1 + u / a.chunk_tiles;
        const int cs = a.ref_tok + (chunk - 1) * a.chunk_tok;
        const int ce = min(cs + a.chunk_tok, a.seq_len);
        split_rows<BM>(cs, ce, (ce - cs + BM - 1) / BM, u % a.chunk_tiles, t.q0, t.q1);
    }
    if (chunk == 0) {
        t.n = 1;
        t.b0 = 0;
        t.e0 = a.ref_tok;
        t.b1 = t.e1 = 0;
    } else {
        const int lo = max(1, chunk - a.window);
        const int end = min(a.ref_tok + chunk * a.chunk_tok, a.seq_len);
        if (lo == 1) {  // c_0 and c_1 are adjacent: one range
            t.n = 1;
            t.b0 = 0;
            t.e0 = end;
            t.b1 = t.e1 = 0;
        } else {
            t.n = 2;
            t.b0 = 0;
            t.e0 = a.ref_tok;
            t.b1 = a.ref_tok + (lo - 1) * a.chunk_tok;
            t.e1 = end;
        }
    }
    return t;
}

__device__ __forceinline__ int range_begin(const AttnArgs& a, const TileRanges& t, int r) {
    return a.mode == 0 ? a.range_begin[r] : (r == 0 ? t.b0 : t.b1);
}
__device__ __forceinline__ int range_end(const AttnArgs& a, const TileRanges& t, int r) {
    return a.mode == 0 ? a.range_end[r] : (r == 0 ? t.e0 : t.e1);
}

__device__ __forceinline__ f32x16_t mfma32x32x16(bf16x8_t a, bf16x8_t b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// ----------------------------------------------------------------------------
// bf16 MFMA kernel
// ----------------------------------------------------------------------------
// LDS holds two K tiles and two V tiles (double buffering), each BN rows of D
// bf16 with no padding. Every 16-byte chunk of a row sits at chunk position
// (chunk ^ swz(row)), which spreads both the K operand reads (same chunk of
// consecutive rows) and the transposing V reads (two adjacent chunks of four
// consecutive rows) over distinct banks. Tiles are filled by direct
// global->LDS loads (global_load_lds_dwordx4): each wave instruction writes
// 1 KB of LDS linearly, so each lane fetches the global chunk that belongs at
// its LDS position (lds_swizzle).

// V^T tile: D rows of 64 keys (128 bytes, 8 chunks of 8 keys). Chunk c of row
// d sits at position c ^ vt_swizzle(d): over any 16 consecutive rows the pair
// (row parity, position) takes all 16 values, so 16 lanes reading the same
// chunk of 16 consecutive rows hit 64 distinct banks.
__device__ __forceinline__ int vt_swizzle(int d) { return (d >> 1) & 7; }




template <int D, bool VT, bool OF32>
__global__ __launch_bounds__(kBf16Threads, 1) void attn_fwd_bf16_kernel(const AttnArgs a) {
    constexpr int BM = kTileRowsBf16;  // query rows per workgroup
    constexpr int BN = 64;             // keys per tile
    constexpr int CPR = D / 8;         // 16-byte chunks per key row
    constexpr int ROWB = D * 2;        // bytes per key row
    constexpr int TILEB = BN * ROWB;
    constexpr int NW = kBf16Threads / 64;            // waves per workgroup, 32 query rows each
    constexpr int NI = TILEB / (kBf16Threads * 16);  // direct loads per thread per tensor per tile
    constexpr int KK = D / 16;  // MFMA k-steps over head_dim
    constexpr int DB = D / 32;  // 32-row blocks of O^T
    constexpr int NK = 2 * KK;  // K fragments per tile = score MFMAs per wave
    constexpr int NV = 4 * DB;  // V fragments per tile = P.V MFMAs per wave
    constexpr int NF = NK + NV;
    constexpr int RING = 4;        // fragments read ahead of their MFMA
    constexpr int EPG = 32 / NK;   // P elements formed per score MFMA
    constexpr int FPG = 32 / NV;   // scores scaled per P.V MFMA
    constexpr int NBUF = 4;        // LDS buffers per tensor (a power of two)
    static_assert(NI * kBf16Threads * 16 == TILEB, "tile must split evenly over the threads");
    static_assert(BM == NW * 32, "one 32-row query block per wave");
    static_assert(NF % RING == 0 && NK >= RING && EPG % 2 == 0, "fragment ring layout");

    // K tile j sits in buffer j % 4 of the first four, V tile j in buffer
    // j % 4 of the last four.
    __shared__ __attribute__((aligned(1024))) unsigned char smem[2 * NBUF * TILEB];
    lds_u8* const L = (lds_u8*)(smem);
    const uint32_t lds_base = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(L));

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int hw = lane >> 5;   // half-wave: which 8-element k-slice a lane feeds
    const int l32 = lane & 31;  // the query column (and operand row) a lane owns

    const int total = a.n_qtiles * a.B * a.H;
    const int id = xcd_logical_id(blockIdx.x, total);
    const int tile = id % a.n_qtiles;
    const int bh = id / a.n_qtiles;
    const int head = bh % a.H;
    const int bat = bh / a.H;
    const TileRanges tr = plan_tile<BM>(a, tile);

    const __bf16* qp = static_cast<const __bf16*>(a.q) + bat * a.q_sb + head * a.q_sh;
    const __bf16* kp = static_cast<const __bf16*>(a.k) + bat * a.k_sb + head * a.k_sh;
    const __bf16* vp = static_cast<const __bf16*>(a.v) + bat * a.v_sb + head * a.v_sh;

    // ---- key tiles: the tiles of range 0, then those of range 1, ... Tile j
    // of the walk (clamped to the last tile) is found by counting tiles per
    // range; this runs only at range boundaries.
    struct KeyTile {
        int k0, ke;
    };
    auto range_tiles = [&](int r) { return (range_end(a, tr, r) - range_begin(a, tr, r) + BN - 1) / BN; };
    int n = 0;
    for (int r = 0; r < tr.n; ++r) n += range_tiles(r);
    auto tile_at = [&](int j) __attribute__((always_inline)) {
        j = min(j, n - 1);
        int r = 0, first = 0;
        while (r + 1 < tr.n && j >= first + range_tiles(r)) {
            first += range_tiles(r);
            ++r;
        }
        return KeyTile{range_begin(a, tr, r) + (j - first) * BN, range_end(a, tr, r)};
    };
    // Smallest tile index >= j whose tile ends its range (the walk's last
    // tile if there is none).
    auto next_range_end = [&](int j) __attribute__((always_inline)) {
        int last = 0;
        for (int r = 0; r < tr.n; ++r) {
            last += range_tiles(r);
            if (last - 1 >= j) return last - 1;
        }
        return n - 1;
    };

    // ---- direct global->LDS loads of one tile. Rows past the range end
    // re-read the range's last row (finite data; its scores are masked). A V^T
    // tile takes, for each dimension d, the 8-key groups of the tile from the
    // cache's V block(s); groups past the range end re-read the group holding
    // the range's last key (its other columns are the append's zeros). Each
    // wave loads NI blocks of 1 KB per tensor. The lane offsets from the
    // tile's scalar base are the same for every tile of a range except its
    // last, so they are planned again only for a range's last tile and for the
    // tile after it.
    auto plan = [&](uint32_t (&off)[NI], bool is_v, const KeyTile& t) __attribute__((always_inline)) {
        // the thread index read afresh: the per-lane terms below are then
        // recomputed on this rare path instead of being kept live (spilled)
        // across the key loop
        const int tix = fresh_thread_index();
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const int ch = i * kBf16Threads + tix;
            if (!is_v || !VT) {
                const int row = min(ch / CPR, t.ke - 1 - t.k0);
                const int gc = (ch % CPR) ^ lds_swizzle<D>(ch / CPR);
                const int64_t st = is_v ? a.v_st : a.k_st;
                off[i] = static_cast<uint32_t>((row * st + gc * 8) * 2);
            } else {
                const int d = ch >> 3;
                const int b0 = t.k0 & ~63;  // first cache block of the tile
                const int g = min(t.k0 + 8 * ((ch & 7) ^ vt_swizzle(d)), (t.ke - 1) & ~7) - b0;
                off[i] = static_cast<uint32_t>(((g >> 6) * (64 * D) + d * 64 + (g & 63)) * 2);
            }
        }
    };
    const uint32_t lds_wave = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(wave * 1024));
    // Byte offsets of K buffer j % 4 from the start of LDS, and of V buffer
    // j % 4 from the start of the V buffers (NBUF * TILEB further on).
    auto kbuf = [](int j) { return static_cast<uint32_t>((j & (NBUF - 1)) * TILEB); };
    auto vbuf = [](int j) { return static_cast<uint32_t>((j & (NBUF - 1)) * TILEB); };
    auto kbase = [&](const KeyTile& t) { return uniform_ptr(kp + static_cast<int64_t>(t.k0) * a.k_st); };
    auto vbase = [&](const KeyTile& t) {
        return VT ? uniform_ptr(vp + static_cast<int64_t>(t.k0 & ~63) * D)
                  : uniform_ptr(vp + static_cast<int64_t>(t.k0) * a.v_st);
    };
    // Load i (0 <= i < NI) of two tiles issued together: source p0 + lane
    // offset o0 into LDS byte offset l0, and likewise p1, o1, l1.
    auto dma_pair = [&](int i, const void* p0, uint32_t o0, uint32_t l0, const void* p1, uint32_t o1,
                        uint32_t l1) __attribute__((always_inline)) {
        const uint32_t blk = lds_base + lds_wave + i * NW * 1024;
        lds_dma16x2(p0, o0, l0 + blk, p1, o1, l1 + blk);
    };

    // ---- Q^T operand (B of the score MFMA): lane holds q[row][16*kk + 8*hw .. +8].
    const int qrow = tr.q0 + wave * 32 + l32;
    const bool row_ok = qrow < tr.q1;
    bf16x8_t qf[KK];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
        if (row_ok) {
            qf[kk] = *reinterpret_cast<const bf16x8_t*>(qp + qrow * a.q_st + kk * 16 + hw * 8);
        } else {
            qf[kk] = bf16x8_t{};
        }
    }
    // The Q loads land before any direct load is issued, so no wait that the
    // compiler places for them can be miscounted.
    wait_lds_dma();

    // ---- per-lane LDS byte offsets of the operand fragments within a tile.
    // K fragment (kk, kb): row l32 + 32*kb (permuted with VT), chunk 2*kk + hw.
    const int k_row = VT ? k_perm(l32) : l32;
    const int k_swz = lds_swizzle<D>(k_row);
    uint32_t koff[KK];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) koff[kk] = k_row * ROWB + (((2 * kk + hw) ^ k_swz) << 4);
    // V fragment (j, d): with VT, row 32*d + l32 of the V^T tile, keys
    // 16*j + 8*hw .. + 7; else two transposing reads of the row-major tile,
    // rows 16*j + 4*hw + gi/4 (and + 8), element columns 32*d + 16*(grp & 1) +
    // 4*(gi & 3).
    constexpr int kVtRowBytes = 64 * 2;  // a V^T row: 64 keys
    const int grp = lane >> 4, gi = lane & 15;
    const int v_row = 4 * hw + (gi >> 2);
    const int v_swz_lo = lds_swizzle<D>(v_row), v_swz_hi = lds_swizzle<D>(v_row + 8);
    const int v_cbase = 2 * (grp & 1) + ((gi & 3) >> 1);
    const int v_half = (gi & 1) * 8;
    uint32_t voff[VT ? 4 : 2 * DB];
    if constexpr (VT) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
            voff[j] = NBUF * TILEB + l32 * kVtRowBytes + (((2 * j + hw) ^ vt_swizzle(l32)) << 4);
    } else {
#pragma unroll
        for (int d = 0; d < DB; ++d) {
            const int cc = 4 * d + v_cbase;
            voff[2 * d] = NBUF * TILEB + v_row * ROWB + ((cc ^ v_swz_lo) << 4) + v_half;
            voff[2 * d + 1] = NBUF * TILEB + (v_row + 8) * ROWB + ((cc ^ v_swz_hi) << 4) + v_half;
        }
    }
    // Fragment s of a tile's stream: K fragments 0..NK-1 (kk = s/2, kb = s%2)
    // from the K buffer at byte offset kb_off, then V fragments
    // (j = (s-NK)/DB, d = (s-NK)%DB) from the V buffer at vb_off. Lane offset
    // plus a constant: the buffer offsets fold into the read's immediate.
    auto read_frag = [&](int s, uint32_t kb_off, uint32_t vb_off) __attribute__((always_inline)) {
        bf16x8_t f;
        if (s < NK) {
            const int kk = s >> 1, kb = s & 1;
            f = *reinterpret_cast<const lds_bf16x8_t*>(L + koff[kk] + (kb_off + kb * 32 * ROWB));
        } else {
            const int j = (s - NK) / DB, d = (s - NK) % DB;
            if constexpr (VT) {
                f = *reinterpret_cast<const lds_bf16x8_t*>(L + voff[j] + (vb_off + d * 32 * kVtRowBytes));
            } else {
                const bf16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
                    (lds_bf16x4_t*)(L + voff[2 * d] + (vb_off + 16 * j * ROWB)));
                const bf16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
                    (lds_bf16x4_t*)(L + voff[2 * d + 1] + (vb_off + 16 * j * ROWB)));
                f = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
            }
        }
        return f;
    };

    // ---- state
    f32x16_t acc[DB];
#pragma unroll
    for (int i = 0; i < DB; ++i) acc[i] = f32x16_t{};
    float m_run;            // running max in the scaled log2 domain (lazy)
    float l_run = 0.f;      // this lane's partial row sum
    const float c = a.scale_log2;
    // S^T output layout: register i of block kb holds key 32*kb + (VT ?
    // 16*(i/8) + 8*hw + i%8 : 8*(i/4) + 4*hw + i%4) of the tile, query l32.
    auto key_of = [&](int kb, int i) {
        return 32 * kb + (VT ? 16 * (i / 8) + 8 * hw + (i % 8) : 8 * (i / 4) + 4 * hw + (i % 4));
    };
    auto mask_tile = [&](f32x16_t (&s)[2], const KeyTile& kt) __attribute__((always_inline)) {
        if (kt.k0 + BN > kt.ke) {
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 16; ++i)
                    if (kt.k0 + key_of(kb, i) >= kt.ke) s[kb][i] = kNegInf;
        }
    };
    // Largest score of this query in the tile (both half-waves).
    auto row_max = [&](const f32x16_t (&s)[2]) __attribute__((always_inline)) {
        float mx = fmaxf(s[0][0], s[1][0]);
#pragma unroll
        for (int i = 1; i < 16; ++i) mx = fmaxf(mx, fmaxf(s[0][i], s[1][i]));
        const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
        return fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
    };
    // P = exp2(x) for elements [e, e + 2) of x, rounded to bf16 into its P^T
    // operand slot (k-step e/8, slot e%8); the fp32 values are summed into *lt.
    // (Summing the rounded pair with v_dot2_f32_bf16 instead costs more: that
    // instruction waits for the MFMA in flight, a plain fp32 add does not.)
    auto form_p2 = [&](const f32x16_t (&x)[2], bf16x8_t (&pf)[4], int e, float& lt) __attribute__((always_inline)) {
        const float p0 = __builtin_amdgcn_exp2f(x[e >> 4][e & 15]);
        const float p1 = __builtin_amdgcn_exp2f(x[(e + 1) >> 4][(e + 1) & 15]);
        pf[e >> 3][e & 7] = static_cast<__bf16>(p0);
        pf[e >> 3][(e & 7) + 1] = static_cast<__bf16>(p1);
        lt += p0 + p1;
    };

    // ---- prologue: tiles 0..3 of K and 0..1 of V in flight, S(0) and its
    // exact maximum (the lazy running max starts from it), x(0) = S(0)*c - m.
    uint32_t offk[NI], offv[NI];  // lane offsets of the loads of the current K and V tiles
    {
        const KeyTile k0t = tile_at(0), k1t = tile_at(1), k2t = tile_at(2), k3t = tile_at(3);
        uint32_t o0[NI], o1[NI];
        plan(o0, false, k0t);
        plan(o1, true, k0t);
#pragma unroll
        for (int i = 0; i < NI; ++i)
            dma_pair(i, kbase(k0t), o0[i], kbuf(0), vbase(k0t), o1[i], NBUF * TILEB + vbuf(0));
        plan(o0, false, k1t);
        plan(o1, true, k1t);
#pragma unroll
        for (int i = 0; i < NI; ++i)
            dma_pair(i, kbase(k1t), o0[i], kbuf(1), vbase(k1t), o1[i], NBUF * TILEB + vbuf(1));
        plan(o0, false, k2t);
        plan(o1, false, k3t);
#pragma unroll
        for (int i = 0; i < NI; ++i) dma_pair(i, kbase(k2t), o0[i], kbuf(2), kbase(k3t), o1[i], kbuf(3));
    }
    wait_lds_dma();
    __syncthreads();

    // A wave whose 32 query rows all lie past the tile's end (the last query
    // tile of a chunk) takes part in the loads and barriers only.
    const bool busy = __builtin_amdgcn_readfirstlane(static_cast<int>(tr.q0 + wave * 32 < tr.q1)) != 0;
    f32x16_t xa[2], xb[2];  // x(t) and S(t+1) / x(t+1), alternating roles
    m_run = 0.f;
    if (busy) {
        bf16x8_t kf[NK];
#pragma unroll
        for (int s = 0; s < NK; ++s) kf[s] = read_frag(s, kbuf(0), vbuf(0));
        xa[0] = xa[1] = f32x16_t{};
#pragma unroll
        for (int s = 0; s < NK; ++s) xa[s & 1] = mfma32x32x16(kf[s], qf[s >> 1], xa[s & 1]);
        mask_tile(xa, tile_at(0));
        m_run = row_max(xa) * c;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int i = 0; i < 16; ++i) xa[kb][i] = fmaf(xa[kb][i], c, -m_run);
    }
    bf16x8_t fr[RING];
#pragma unroll
    for (int s = 0; s < RING; ++s) fr[s] = read_frag(s, kbuf(1), vbuf(1));
    // Iteration 0 loads K(4) into the buffer of K(0), and a wave without rows
    // reaches that load at once: every wave must be done reading K(0) first.
    __syncthreads();

    // ---- main loop: iteration t, with x = x(t) and nx receiving S(t+1).
    // Stage 1: the score MFMAs of tile t+1, each with its share of P(t)
    // (exp2, bf16, row sum). Check: if some lane's row sum of the tile
    // exceeds 2^16 (a score more than 16 above the running max in the log2
    // domain, or a non-finite value), raise the max to the tile's maximum,
    // rescale O and the row sum, and form P(t) again. Stage 2: the P.V MFMAs
    // of tile t, each with its share of x(t+1) = S(t+1)*c - m. Every MFMA is
    // preceded by the LDS read of the fragment RING MFMAs ahead; tile t+4 of
    // K and tile t+2 of V are loaded during stage 2. At the end each wave
    // waits for its loads of the previous iteration and the barrier publishes
    // K(t+2), K(t+3) and V(t+1).
    //
    // Tiles t+1 (scores), t+2 (V load) and t+4 (K load) move one tile on in
    // their range unless a tile among t+1..t+4 ends a range; only then (at
    // most a few iterations per range, and at the end of the walk) are they
    // looked up afresh, the load offsets planned again and the mask of tile
    // t+1 decided.
    int event = 0;                 // smallest range-ending tile index >= the last refresh's t + 2
    const void* kptr = nullptr;    // K source of tile t+4
    const void* vptr = nullptr;    // V source of tile t+2
    KeyTile ks{0, BN};             // tile t+1 when it ends its range (scores to mask)
    bool mask_next = false;
    const int64_t kstep = static_cast<int64_t>(BN) * a.k_st * 2;  // bytes per tile of keys
    const int64_t vstep = static_cast<int64_t>(BN) * (VT ? D : a.v_st) * 2;
    auto refresh = [&](int t) __attribute__((always_inline)) {
        if (__builtin_expect(t + 4 >= event, 0)) {
            const KeyTile k4 = tile_at(t + 4), v2 = tile_at(t + 2);
            ks = tile_at(t + 1);
            mask_next = ks.k0 + BN > ks.ke;
            plan(offk, false, k4);
            plan(offv, true, v2);
            kptr = kbase(k4);
            vptr = vbase(v2);
            event = __builtin_amdgcn_readfirstlane(next_range_end(t + 2));
            // The range bounds may come from scalar loads, which share a
            // counter with the LDS reads and complete out of order: wait for
            // them here, on this rare path, so that no full wait lands on the
            // common path where fragment reads are still in flight.
            wait_lds_reads<0>();
        } else {
            kptr = static_cast<const char*>(kptr) + kstep;
            vptr = static_cast<const char*>(vptr) + vstep;
            mask_next = false;
        }
    };
    // The barrier orders only this workgroup's LDS use: the compiler may not
    // move LDS accesses across it, and no wait is needed for the fragment
    // reads still in flight (their buffer is not written next).
    auto end_tile = [&]() __attribute__((always_inline)) {
        wait_lds_dma_but<2 * NI>();
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
    };
    auto iteration = [&](int u, int t, f32x16_t (&x)[2], f32x16_t (&nx)[2]) __attribute__((always_inline)) {
        const uint32_t kb1 = kbuf(u + 1), kb2 = kbuf(u + 2), vb0 = vbuf(u);
        refresh(t);
        bf16x8_t pf[4];
        float lt0 = 0.f, lt1 = 0.f;
        nx[0] = nx[1] = f32x16_t{};
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int g = 0; g < NK; ++g) {
            nx[g & 1] = mfma32x32x16(fr[g % RING], qf[g >> 1], nx[g & 1]);
            fr[g % RING] = read_frag(g + RING, kb1, vb0);
#pragma unroll
            for (int e = EPG * g; e < EPG * (g + 1); e += 2) form_p2(x, pf, e, (e & 2) ? lt1 : lt0);
            __builtin_amdgcn_sched_barrier(0);
        }
        if (__builtin_expect(__any(!(lt0 + lt1 <= 0x1p16f)), 0)) {
            const float dm = fmaxf(row_max(x), 0.f);
            const float alpha = __builtin_amdgcn_exp2f(-dm);
            m_run += dm;
            l_run *= alpha;
#pragma unroll
            for (int d = 0; d < DB; ++d) acc[d] *= alpha;
            lt0 = lt1 = 0.f;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 16; ++i) x[kb][i] -= dm;
#pragma unroll
            for (int e = 0; e < 32; e += 2) form_p2(x, pf, e, (e & 2) ? lt1 : lt0);
        }
        l_run += lt0 + lt1;
        if (mask_next) mask_tile(nx, ks);
        const float nm = -m_run;
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int k = 0; k < NV; ++k) {
            acc[k % DB] = mfma32x32x16(fr[(NK + k) % RING], pf[k / DB], acc[k % DB]);
            fr[(NK + k) % RING] = read_frag((NK + k + RING) % NF, NK + k + RING < NF ? kb1 : kb2, vb0);
#pragma unroll
            for (int e = FPG * k; e < FPG * (k + 1); ++e) nx[e >> 4][e & 15] = pin(fmaf(nx[e >> 4][e & 15], c, nm));
            if (k % (NV / NI) == NV / (2 * NI)) {
                const int i = k / (NV / NI);
                dma_pair(i, kptr, offk[i], kbuf(u), vptr, offv[i], NBUF * TILEB + vbuf(u + 2));
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        end_tile();
    };
    if (busy) {
        for (int t = 0; t < n; t += 4) {
            iteration(0, t, xa, xb);
            if (t + 1 >= n) break;
            iteration(1, t + 1, xb, xa);
            if (t + 2 >= n) break;
            iteration(2, t + 2, xa, xb);
            if (t + 3 >= n) break;
            iteration(3, t + 3, xb, xa);
        }
    } else {
        // the same loads and barriers, no arithmetic
        for (int t = 0; t < n; ++t) {
            refresh(t);
#pragma unroll
            for (int i = 0; i < NI; ++i)
                dma_pair(i, kptr, offk[i], kbuf(t), vptr, offv[i], NBUF * TILEB + vbuf(t + 2));
            end_tile();
        }
    }
    wait_lds_dma();  // no load may still be writing LDS when the workgroup ends

    // ---- epilogue: normalise, store rows inside the tile, rounded to bf16
    // (nearest even) or, with OF32, as the fp32 values that rounding would take
    const float l_tot = l_run + __shfl_xor(l_run, 32);
    const float inv = 1.f / l_tot;
    if (row_ok) {
        const int64_t orow = bat * a.o_sb + head * a.o_sh + qrow * a.o_st;
#pragma unroll
        for (int d = 0; d < DB; ++d) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                if constexpr (OF32) {
                    float4 w;
                    w.x = acc[d][4 * g + 0] * inv;
                    w.y = acc[d][4 * g + 1] * inv;
                    w.z = acc[d][4 * g + 2] * inv;
                    w.w = acc[d][4 * g + 3] * inv;
                    *reinterpret_cast<float4*>(static_cast<float*>(a.o) + orow + 32 * d + 8 * g + 4 * hw) = w;
                } else {
                    bf16x4_t w;
#pragma unroll
                    for (int e = 0; e < 4; ++e) w[e] = static_cast<__bf16>(acc[d][4 * g + e] * inv);
                    *reinterpret_cast<bf16x4_t*>(static_cast<__bf16*>(a.o) + orow + 32 * d + 8 * g + 4 * hw) = w;
                }
            }
        }
        if (a.lse != nullptr && hw == 0) {
            a.lse[(static_cast<int64_t>(bat) * a.H + head) * a.Lq + qrow] =
                (m_run + __log2f(l_tot)) * 0.69314718055994530942f;
        }
    }
}

// ----------------------------------------------------------------------------
// fp32 VALU kernel (small problems, exact fp32 arithmetic)
// ----------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void attn_fwd_f32_kernel(const AttnArgs a) {
    constexpr int BM = kTileRowsF32;  // 64 query rows, 4 lanes each
    constexpr int BN = 32;
    constexpr int DP = D / 4;         // elements per lane
    constexpr int PSTR = DP + 1;      // padded quarter-row pitch in LDS
    constexpr int RSTR = 4 * PSTR;
    constexpr int C4 = D / 4;         // float4 per key row

    __shared__ float Ks[BN * RSTR];
    __shared__ float Vs[BN * RSTR];

    const int tid = threadIdx.x;
    const int row = tid >> 2, part = tid & 3;
    const int total = a.n_qtiles * a.B * a.H;
    const int id = xcd_logical_id(blockIdx.x, total);
    const int tile = id % a.n_qtiles;
    const int bh = id / a.n_qtiles;
    const int head = bh % a.H;
    const int bat = bh / a.H;
    const TileRanges tr = plan_tile<BM>(a, tile);

    const float* qp = static_cast<const float*>(a.q) + bat * a.q_sb + head * a.q_sh;
    const float* kp = static_cast<const float*>(a.k) + bat * a.k_sb + head * a.k_sh;
    const float* vp = static_cast<const float*>(a.v) + bat * a.v_sb + head * a.v_sh;
    const int qrow = tr.q0 + row;
    const bool row_ok = qrow < tr.q1;

    float qv[DP], ov[DP];
#pragma unroll
    for (int e = 0; e < DP; ++e) {
        qv[e] = row_ok ? qp[qrow * a.q_st + part * DP + e] : 0.f;
        ov[e] = 0.f;
    }
    float m = kNegInf, l = 0.f;
    const float c = a.scale_log2;

    for (int r = 0; r < tr.n; ++r) {
        const int kb = range_begin(a, tr, r), ke = range_end(a, tr, r);
        for (int k0 = kb; k0 < ke; k0 += BN) {
            __syncthreads();
            for (int ch = tid; ch < BN * C4; ch += 256) {
                const int kr = ch / C4, c4 = ch % C4;
                float4 kv = make_float4(0.f, 0.f, 0.f, 0.f), vv = kv;
                if (k0 + kr < ke) {
                    kv = *reinterpret_cast<const float4*>(kp + (k0 + kr) * a.k_st + c4 * 4);
                    if (!a.v_blocked)
                        vv = *reinterpret_cast<const float4*>(vp + (k0 + kr) * a.v_st + c4 * 4);
                }
                const int d0 = c4 * 4;
                const int base = kr * RSTR + (d0 / DP) * PSTR + d0 % DP;
                Ks[base + 0] = kv.x; Ks[base + 1] = kv.y; Ks[base + 2] = kv.z; Ks[base + 3] = kv.w;
                if (!a.v_blocked) {
                    Vs[base + 0] = vv.x; Vs[base + 1] = vv.y; Vs[base + 2] = vv.z; Vs[base + 3] = vv.w;
                }
            }
            if (a.v_blocked) {
                // Dimension-major cache blocks: element (key, d) sits at
                // (key / 64) * 64 * D + d * 64 + key % 64.
                for (int e = tid; e < BN * D; e += 256) {
                    const int d = e / BN, kr = e % BN, key = k0 + kr;
                    Vs[kr * RSTR + (d / DP) * PSTR + d % DP] =
                        key < ke ? vp[(key >> 6) * (64 * D) + d * 64 + (key & 63)] : 0.f;
                }
            }
            __syncthreads();
            const int n = min(BN, ke - k0);
            for (int j = 0; j < n; ++j) {
                const float* kr = &Ks[j * RSTR + part * PSTR];
                float dot = 0.f;
#pragma unroll
                for (int e = 0; e < DP; ++e) dot = fmaf(qv[e], kr[e], dot);
                dot += __shfl_xor(dot, 1);
                dot += __shfl_xor(dot, 2);
                const float s = dot * c;
                const float m_new = fmaxf(m, s);
                const float alpha = exp2f(m - m_new);
                const float p = exp2f(s - m_new);
                l = fmaf(l, alpha, p);
                const float* vr = &Vs[j * RSTR + part * PSTR];
#pragma unroll
                for (int e = 0; e < DP; ++e) ov[e] = fmaf(ov[e], alpha, p * vr[e]);
                m = m_new;
            }
        }
    }

    if (row_ok) {
        float* op = static_cast<float*>(a.o) + bat * a.o_sb + head * a.o_sh + qrow * a.o_st;
        const float inv = 1.f / l;
#pragma unroll
        for (int e = 0; e < DP; ++e) op[part * DP + e] = ov[e] * inv;
        if (a.lse != nullptr && part == 0) {
            a.lse[(static_cast<int64_t>(bat) * a.H + head) * a.Lq + qrow] =
                (m + log2f(l)) * 0.69314718055994530942f;
        }
    }
}

template <int D, bool VT>
void launch_bf16_out(const AttnArgs& a, dim3 grid, dim3 block, hipStream_t s) {
    if (a.o_f32) hipLaunchKernelGGL((attn_fwd_bf16_kernel<D, VT, true>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((attn_fwd_bf16_kernel<D, VT, false>), grid, block, 0, s, a);
}

}  // namespace

hipError_t launch_attn_bf16(const AttnArgs& a, int head_dim, hipStream_t s) {
    const dim3 grid(a.n_qtiles * a.B * a.H), block(kBf16Threads);
    if (head_dim == 128) {
        if (a.v_blocked) launch_bf16_out<128, true>(a, grid, block, s);
        else launch_bf16_out<128, false>(a, grid, block, s);
    } else if (head_dim == 64) {
        if (a.v_blocked) launch_bf16_out<64, true>(a, grid, block, s);
        else launch_bf16_out<64, false>(a, grid, block, s);
    } else {
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_attn_f32(const AttnArgs& a, int head_dim, hipStream_t s) {
    const dim3 grid(a.n_qtiles * a.B * a.H), block(256);
    if (head_dim == 128) {
        hipLaunchKernelGGL(attn_fwd_f32_kernel<128>, grid, block, 0, s, a);
    } else if (head_dim == 64) {
        hipLaunchKernelGGL(attn_fwd_f32_kernel<64>, grid, block, 0, s, a);
    } else {
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace tmk
