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
// Per 64-key tile:
//   S^T (keys x queries) = K Q^T with v_mfma_f32_32x32x16_bf16, K from LDS,
//     Q^T held in registers for the whole loop;
//   online softmax in fp32 on the MFMA output layout, where each lane owns one
//     query column and half of its keys; exp2 with the scale folded in, and a
//     lazily-updated running max (the accumulator is only rescaled when the
//     max grows by more than 2^8, which keeps P <= 256);
//   O^T (head_dim x queries) += V^T P^T with the same MFMA, P^T straight from
//     registers (bf16, rounded to nearest even). From the KV cache, whose V
//     blocks are stored dimension-major, the V tile lands in LDS as V^T and
//     each operand is one 16-byte read; the K rows are fed to the S MFMA in a
//     permuted order that makes each lane's P^T elements 8 consecutive keys.
//     From row-major V (whole-sequence calls on caller tensors) the operand is
//     read with the gfx950 transposing LDS read.
// K/V tiles are double-buffered in LDS and filled by direct global->LDS loads,
// so the next tile's loads are in flight while the current tile is computed.
//
// fp32 kernel: a plain VALU kernel (4 lanes per query row, exact running max)
// for fp32 inputs; it exists for correctness at small sizes.

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "tm_internal.h"

namespace tmk {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) bf16x4_t lds_bf16x4_t;

constexpr float kNegInf = -__builtin_inff();
// Threads per workgroup of the bf16 kernel: 8 waves (two per SIMD) sharing
// every K/V tile staged in LDS.
constexpr int kBf16Threads = 512;
// s_waitcnt immediate (gfx9 encoding) for vmcnt(0), expcnt and lgkmcnt unconstrained.
constexpr int kWaitVmcnt0 = 0x0F70;

// 32-bit LDS byte address of a __shared__ object, made wave-uniform.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    const uint32_t a = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(
        (const __attribute__((address_space(3))) unsigned char*)(p)));
    return __builtin_amdgcn_readfirstlane(a);
}

// A pointer that is the same in every lane, held in scalar registers.
__device__ __forceinline__ const void* uniform_ptr(const void* p) {
    const uint64_t v = reinterpret_cast<uint64_t>(p);
    const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v));
    const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v >> 32));
    return reinterpret_cast<const void*>((static_cast<uint64_t>(hi) << 32) | lo);
}

// Two direct global->LDS loads (global_load_lds_dwordx4) of 16 bytes per lane:
// load n reads from the wave-uniform base sbase<n> plus the lane's byte offset
// voff<n>, and lane l's bytes land at LDS address lds<n> + 16 * l. The LDS
// address goes through M0 (saved and restored); an SALU write of M0 needs one
// wait state before an LDS-DMA instruction (or anything else) reads it, hence
// the s_nop after each write. Written as inline assembly so that these loads
// stay out of the compiler's wait bookkeeping, which would otherwise make LDS
// reads of one tile wait for the loads of later tiles; the kernel waits for
// them explicitly before the barrier that publishes a tile.
__device__ __forceinline__ void lds_dma16x2(const void* sbase0, uint32_t voff0, uint32_t lds0,
                                            const void* sbase1, uint32_t voff1, uint32_t lds1) {
    uint32_t saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %1\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %2, %3\n\t"
        "s_mov_b32 m0, %4\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %5, %6\n\t"
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0"
        : "=&s"(saved)
        : "s"(lds0), "v"(voff0), "s"(sbase0), "s"(lds1), "v"(voff1), "s"(sbase1));
}

// Wait until every direct global->LDS load issued by this wave has written
// LDS. The barrier that publishes a tile only orders LDS operations; the
// direct loads count as vector-memory operations, so each wave waits for its
// own before the barrier, and after the barrier the whole tile is in place.
__device__ __forceinline__ void wait_lds_dma() { __builtin_amdgcn_s_waitcnt(kWaitVmcnt0); }
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

// Workgroups are dispatched round-robin over the 8 XCDs (each with its own L2).
// Renumber them so that consecutive logical ids (the query tiles of one head,
// which stream the same K/V) land on the same XCD.
__device__ __forceinline__ int xcd_logical_id(int bid, int total) {
    constexpr int kXcds = 8;
    const int per = total / kXcds, rem = total % kXcds;
    const int x = bid % kXcds, j = bid / kXcds;
    return x * per + min(x, rem) + j;
}

// Query rows [q0, q1) of tile `tile` and its key ranges. Mode 0 reads the
// ranges from the kernel arguments; mode 1 derives them from the geometry.
struct TileRanges {
    int q0, q1;
    int n;         // number of ranges
    int b0, e0;    // mode 1 ranges (at most two)
    int b1, e1;
};

template <int BM>
__device__ __forceinline__ TileRanges plan_tile(const AttnArgs& a, int tile) {
    TileRanges t;
    if (a.mode == 0) {
        t.q0 = tile * BM;
        t.q1 = min(t.q0 + BM, a.Lq);
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
        t.q0 = nat * BM;
        t.q1 = min(t.q0 + BM, a.ref_tok);
    } else {
        const int u = nat - a.ref_tiles;
        chunk = 1 + u / a.chunk_tiles;
        const int cs = a.ref_tok + (chunk - 1) * a.chunk_tok;
        const int ce = min(cs + a.chunk_tok, a.seq_len);
        t.q0 = cs + (u % a.chunk_tiles) * BM;
        t.q1 = min(t.q0 + BM, ce);
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
// its LDS position.
template <int D>
__device__ __forceinline__ int lds_swizzle(int row) {
    // Low three bits: a permutation of 0..7 over any 8 aligned rows (K reads
    // of one chunk from 8 consecutive rows hit 8 distinct 16-byte bank
    // groups), with bits 1-2 distinct over any 4 aligned rows (the V reads'
    // chunk pairs {p, p^1} of 4 consecutive rows are disjoint). Bit 3 (rows
    // of 16 chunks only) separates rows r and r + 8.
    const int low = 2 * (row & 3) + ((row >> 2) & 1);
    return D == 128 ? low + 8 * ((row >> 3) & 1) : low;
}

// V^T tile: D rows of 64 keys (128 bytes, 8 chunks of 8 keys). Chunk c of row
// d sits at position c ^ vt_swizzle(d): over any 16 consecutive rows the pair
// (row parity, position) takes all 16 values, so 16 lanes reading the same
// chunk of 16 consecutive rows hit 64 distinct banks.
__device__ __forceinline__ int vt_swizzle(int d) { return (d >> 1) & 7; }

// Row of the K tile that feeds S^T row r when V is read as V^T: bits 2 and 3
// of r swapped. The S^T output register i of a lane in half-wave hw then holds
// key 16*(i/8) + 8*hw + i%8 of its 32-key block, so the 8 P^T elements a lane
// feeds to a 16-key MFMA step are 8 consecutive keys.
__device__ __forceinline__ int k_perm(int r) { return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1); }



template <int D, bool VT>
__global__ __launch_bounds__(kBf16Threads, 1) void attn_fwd_bf16_kernel(const AttnArgs a) {
    constexpr int BM = kTileRowsBf16;  // query rows per workgroup
    constexpr int BN = 64;             // keys per tile
    constexpr int CPR = D / 8;         // 16-byte chunks per key row
    constexpr int ROWB = D * 2;        // bytes per key row
    constexpr int TILEB = BN * ROWB;
    constexpr int NW = kBf16Threads / 64;   // waves per workgroup, 32 query rows each
    constexpr int NI = TILEB / (kBf16Threads * 16);  // direct loads per thread per tensor per tile
    constexpr int KK = D / 16;              // MFMA k-steps over head_dim
    constexpr int DB = D / 32;              // 32-row blocks of O^T
    static_assert(NI * kBf16Threads * 16 == TILEB, "tile must split evenly over the threads");
    static_assert(BM == NW * 32, "one 32-row query block per wave");

    // Three K and three V tiles, each its own LDS object so that the compiler
    // can tell a tile being read from the tiles whose loads are in flight.
    __shared__ __attribute__((aligned(1024))) unsigned char k_t0[TILEB], k_t1[TILEB], k_t2[TILEB];
    __shared__ __attribute__((aligned(1024))) unsigned char v_t0[TILEB], v_t1[TILEB], v_t2[TILEB];
    unsigned char* const kbuf[3] = {k_t0, k_t1, k_t2};
    unsigned char* const vbuf[3] = {v_t0, v_t1, v_t2};
    const uint32_t lds_k[3] = {lds_addr(k_t0), lds_addr(k_t1), lds_addr(k_t2)};
    const uint32_t lds_v[3] = {lds_addr(v_t0), lds_addr(v_t1), lds_addr(v_t2)};

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

    // Issue the direct loads of one K tile and one V tile. Rows past the range
    // end re-read the range's last row (finite data; its scores are masked).
    // A V^T tile takes, for each dimension d, the 8-key groups of the tile from
    // the cache's V block(s); groups past the range end re-read the group that
    // holds the range's last key (its other columns are the append's zeros).
    // This wave's share of one tile's direct loads: 2 * NI loads of one 1 KB
    // LDS block each, the first NI for the K tile, the rest for the V tile.
    // Lane offsets from the tile's scalar bases are kept in ld_off; they only
    // change with k0 mod 64 (V^T) or for a range's last tile (rows past the
    // range end re-read its last row, V^T groups past it the group holding
    // its last key), so plan_loads recomputes them only then.
    uint32_t ld_off[2 * NI];
    int ld_o = -1;  // k0 mod 64 that ld_off was planned for; -1 after a last tile
    auto plan_loads = [&](int k0, int ke) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < 2 * NI; ++i) {
            const int ch = ((i % NI) * NW + wave) * 64 + lane;
            if (i < NI || !VT) {
                const int row = min(ch / CPR, ke - 1 - k0);
                const int gc = (ch % CPR) ^ lds_swizzle<D>(ch / CPR);
                const int64_t st = i < NI ? a.k_st : a.v_st;
                ld_off[i] = static_cast<uint32_t>((row * st + gc * 8) * 2);
            } else {
                const int d = ch >> 3;
                const int b0 = k0 & ~63;  // first cache block of the tile
                const int g = min(k0 + 8 * ((ch & 7) ^ vt_swizzle(d)), (ke - 1) & ~7) - b0;
                ld_off[i] = static_cast<uint32_t>(((g >> 6) * (64 * D) + d * 64 + (g & 63)) * 2);
            }
        }
        ld_o = k0 + BN <= ke ? (k0 & 63) : -1;
    };
    auto prepare_loads = [&](int k0, int ke) __attribute__((always_inline)) {
        if (k0 + BN > ke || (k0 & 63) != ld_o) plan_loads(k0, ke);
    };
    // Loads j of the K tile and of the V tile (0 <= j < NI), one 1 KB LDS block
    // each, issued together; ldk, ldv are the LDS byte addresses of the tiles.
    const uint32_t lds_wave = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(wave * 1024));
    auto issue_pair = [&](int j, int k0, uint32_t ldk, uint32_t ldv) __attribute__((always_inline)) {
        const void* kbase = kp + static_cast<int64_t>(k0) * a.k_st;
        const void* vbase = VT ? static_cast<const void*>(vp + static_cast<int64_t>(k0 & ~63) * D)
                               : static_cast<const void*>(vp + static_cast<int64_t>(k0) * a.v_st);
        const uint32_t blk = lds_wave + j * NW * 1024;
        lds_dma16x2(uniform_ptr(kbase), ld_off[j], ldk + blk, uniform_ptr(vbase), ld_off[NI + j],
                    ldv + blk);
    };
    auto issue = [&](int k0, int ke, uint32_t ldk, uint32_t ldv) __attribute__((always_inline)) {
        prepare_loads(k0, ke);
#pragma unroll
        for (int j = 0; j < NI; ++j) issue_pair(j, k0, ldk, ldv);
    };

    // Q^T operand (B of the S^T MFMA): lane holds q[row][16*kk + 8*hw .. +8].
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

    f32x16_t acc[DB];
#pragma unroll
    for (int i = 0; i < DB; ++i) acc[i] = f32x16_t{};
    float m_run = kNegInf;  // running max in the scaled log2 domain
    float l_run = 0.f;      // this lane's partial row sum (its 32 keys per tile)
    const float c = a.scale_log2;

    // Per-lane LDS byte offsets. K operand: row l32 (and l32 + 32), chunk
    // 2*kk + hw. V^T operand via the transposing read: rows 16*j + 4*hw + gi/4
    // (and + 8), element columns 32*d + 16*(grp & 1) + 4*(gi & 3).
    const int k_row = VT ? k_perm(l32) : l32;
    const int k_row_off = k_row * ROWB;
    const int k_swz = lds_swizzle<D>(k_row);
    const int grp = lane >> 4, gi = lane & 15;
    const int v_row = 4 * hw + (gi >> 2);
    const int v_swz_lo = lds_swizzle<D>(v_row), v_swz_hi = lds_swizzle<D>(v_row + 8);
    const int v_cbase = 2 * (grp & 1) + ((gi & 3) >> 1);
    const int v_half = (gi & 1) * 8;
    constexpr int kVtRowBytes = 64 * 2;  // a V^T row: 64 keys
    int vt_off[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) vt_off[j] = l32 * kVtRowBytes + (((2 * j + hw) ^ vt_swizzle(l32)) << 4);

    // One tile: keys [k0, ke) from buffers kb, vb. The loads of the next tile
    // (keys from nk0 into nkd, nvd) are spread over the score MFMAs, so that
    // no wave stalls on a full load queue while the others also issue theirs.
    constexpr int kAhead = 4;  // LDS operand reads run this many MFMAs ahead
    auto compute = [&](const unsigned char* kb, const unsigned char* vb, int k0, int ke, int nk0,
                       int nke, uint32_t nkd, uint32_t nvd) __attribute__((always_inline)) {
        // ---- S^T = K Q^T: two 32-key blocks x 32 queries per wave
        f32x16_t s0 = f32x16_t{}, s1 = f32x16_t{};
        constexpr int kLoadEvery = KK / NI;  // k-steps between two load pairs
        static_assert(kLoadEvery >= 1 && kLoadEvery * NI == KK, "loads must spread evenly");
        // K fragments are read in batches of four (two k-steps), one batch
        // ahead; one explicit wait per batch covers its four MFMAs.
        bf16x8_t kf[2 * KK];
        auto read_k = [&](int bt) __attribute__((always_inline)) {
#pragma unroll
            for (int kk = 2 * bt; kk < 2 * bt + 2; ++kk) {
                const int off = k_row_off + (((2 * kk + hw) ^ k_swz) << 4);
                kf[2 * kk] = *reinterpret_cast<const bf16x8_t*>(kb + off);
                kf[2 * kk + 1] = *reinterpret_cast<const bf16x8_t*>(kb + off + 32 * ROWB);
            }
        };
        constexpr int KB = KK / 2;  // batches
        read_k(0);
        if (KB > 1) read_k(1);
#pragma unroll
        for (int bt = 0; bt < KB; ++bt) {
            if (bt + 1 < KB) wait_lds_reads<4>(); else wait_lds_reads<0>();
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int kk = 2 * bt; kk < 2 * bt + 2; ++kk) {
                s0 = mfma32x32x16(kf[2 * kk], qf[kk], s0);
                s1 = mfma32x32x16(kf[2 * kk + 1], qf[kk], s1);
                if (kk % kLoadEvery == 0) issue_pair(kk / kLoadEvery, nk0, nkd, nvd);
            }
            if (bt + 2 < KB) read_k(bt + 2);
            __builtin_amdgcn_sched_barrier(0);
        }

        // Output layout: register i of a lane holds S^T row 8*(i/4) + 4*hw + i%4,
        // i.e. key 16*(i/8) + 8*hw + i%8 with the permuted K rows.
        if (k0 + BN > ke) {
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int kr = k0 + (VT ? 16 * (i / 8) + 8 * hw + (i % 8)
                                        : 8 * (i / 4) + 4 * hw + (i % 4));
                if (kr >= ke) s0[i] = kNegInf;
                if (kr + 32 >= ke) s1[i] = kNegInf;
            }
        }

        // ---- online softmax against the running max m_run, which is shared
        // by the two half-waves holding a query's scores. The common path takes
        // no maximum: P = exp2(S * c - m_run) is formed against the current
        // m_run and kept unless some lane's sum of its 32 values exceeds 2^16
        // (or is not finite), i.e. unless a score exceeds m_run by more than 16
        // in the log2 domain. Otherwise (always on the first tile, rarely
        // after) the exact maximum of both halves is taken, O and the row sum
        // are rescaled and P is formed again. P is at most 2^16 either way, so
        // it and O keep their full relative precision far from overflow.
        bf16x8_t pf[4];
        const bf16x2_t ones = {static_cast<__bf16>(1.f), static_cast<__bf16>(1.f)};
        auto form_p = [&](float neg_m) __attribute__((always_inline)) -> float {
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                pf[i / 8][i % 8] = static_cast<__bf16>(__builtin_amdgcn_exp2f(fmaf(s0[i], c, neg_m)));
                pf[2 + i / 8][i % 8] = static_cast<__bf16>(__builtin_amdgcn_exp2f(fmaf(s1[i], c, neg_m)));
            }
            // Row sum of the bf16-rounded P that is multiplied into V.
            float l = 0.f;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const bf16x2_t pp = {pf[j][2 * e], pf[j][2 * e + 1]};
                    l = __builtin_amdgcn_fdot2_f32_bf16(pp, ones, l, false);
                }
            }
            return l;
        };
        float lt = form_p(-m_run);
        if (__any(!(lt <= 0x1p16f))) {
            float mx = s0[0];
#pragma unroll
            for (int i = 1; i < 16; ++i) mx = fmaxf(mx, s0[i]);
#pragma unroll
            for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s1[i]);
            const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx),
                                                             __float_as_uint(mx), false, false);
            mx = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));  // both halves
            const float m_new = fmaxf(m_run, mx * c);
            const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
            m_run = m_new;
            l_run *= alpha;
#pragma unroll
            for (int d = 0; d < DB; ++d) acc[d] *= alpha;
            lt = form_p(-m_run);
        }
        l_run += lt;

        // ---- O^T += V^T P^T. P^T k-step j covers S rows 16*j .. 16*j + 15
        // with slot e <-> row 16*j + 4*hw + e (e < 4) or 16*j + 8 + 4*hw + e - 4
        // (e >= 4); the V^T operand reads the same keys, 4 at a time.
        if constexpr (VT) {
            // Row 32*d + l32 of the V^T tile, keys 16*j + 8*hw .. + 7, each
            // fragment read kAhead MFMAs before its MFMA.
            // V fragments in batches of DB (one k-step), one batch ahead, one
            // explicit wait per batch.
            bf16x8_t vf[4 * DB];
            auto read_v = [&](int j) __attribute__((always_inline)) {
#pragma unroll
                for (int d = 0; d < DB; ++d)
                    vf[j * DB + d] = *reinterpret_cast<const bf16x8_t*>(vb + vt_off[j] + d * 32 * kVtRowBytes);
            };
            read_v(0);
            read_v(1);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (j < 3) wait_lds_reads<DB>(); else wait_lds_reads<0>();
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int d = 0; d < DB; ++d) acc[d] = mfma32x32x16(vf[j * DB + d], pf[j], acc[d]);
                if (j + 2 < 4) read_v(j + 2);
                __builtin_amdgcn_sched_barrier(0);
            }
            return;
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
#pragma unroll
            for (int d = 0; d < DB; ++d) {
                const int cc = 4 * d + v_cbase;
                const int lo = (16 * j + v_row) * ROWB + ((cc ^ v_swz_lo) << 4) + v_half;
                const int hi = (16 * j + v_row + 8) * ROWB + ((cc ^ v_swz_hi) << 4) + v_half;
                const bf16x4_t vlo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)(vb + lo));
                const bf16x4_t vhi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)(vb + hi));
                const bf16x8_t vf = __builtin_shufflevector(vlo, vhi, 0, 1, 2, 3, 4, 5, 6, 7);
                acc[d] = mfma32x32x16(vf, pf[j], acc[d]);
            }
        }
    };

    // Triple-buffered main loop, unrolled by three so each buffer is named
    // statically: tile t sits in buffer t % 3 and is computed while tiles t+1
    // and t+2 load (the loads of tile t+2 are issued during tile t, into the
    // buffer of tile t-1, which every wave finished before the barrier at the
    // top of iteration t). Past the last tile the loads re-read the last tile
    // (harmless; no one reads those buffers again), which keeps the code free
    // of branches. Each wave issues 2 * NI loads per tile, so waiting until
    // at most 2 * NI are outstanding leaves only tile t+1's in flight.
    struct KeyTile {
        int r, k0, ke;
    };
    auto advance = [&](KeyTile t) __attribute__((always_inline)) {
        KeyTile u = t;
        u.k0 += BN;
        if (u.k0 >= u.ke) {
            if (u.r + 1 >= tr.n) return t;  // past the end: stay on the last tile
            u.r += 1;
            u.k0 = range_begin(a, tr, u.r);
            u.ke = range_end(a, tr, u.r);
        }
        return u;
    };
    int n = 0;
    for (int r = 0; r < tr.n; ++r) n += (range_end(a, tr, r) - range_begin(a, tr, r) + BN - 1) / BN;
    KeyTile cur{0, range_begin(a, tr, 0), range_end(a, tr, 0)};
    KeyTile ld1 = advance(cur);  // tile t+1
    issue(cur.k0, cur.ke, lds_k[0], lds_v[0]);
    issue(ld1.k0, ld1.ke, lds_k[1], lds_v[1]);
    KeyTile ld2 = advance(ld1);  // tile t+2
    auto step = [&](int b) __attribute__((always_inline)) {
        prepare_loads(ld2.k0, ld2.ke);
        wait_lds_dma_but<2 * NI>();
        __syncthreads();  // tile t is in buffer b for every wave
        const int bn = b == 0 ? 2 : b - 1;  // (t + 2) % 3
        compute(kbuf[b], vbuf[b], cur.k0, cur.ke, ld2.k0, ld2.ke, lds_k[bn], lds_v[bn]);
        cur = ld1;
        ld1 = ld2;
        ld2 = advance(ld2);
    };
    for (int t = 0; t < n; t += 3) {
        step(0);
        if (t + 1 >= n) break;
        step(1);
        if (t + 2 >= n) break;
        step(2);
    }
    wait_lds_dma();  // no load may still be writing LDS when the workgroup ends

    // ---- epilogue: normalise, round to bf16, store rows inside the tile
    const float l_tot = l_run + __shfl_xor(l_run, 32);
    const float inv = 1.f / l_tot;
    if (row_ok) {
        __bf16* op = static_cast<__bf16*>(a.o) + bat * a.o_sb + head * a.o_sh + qrow * a.o_st;
#pragma unroll
        for (int d = 0; d < DB; ++d) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                bf16x4_t w;
#pragma unroll
                for (int e = 0; e < 4; ++e) w[e] = static_cast<__bf16>(acc[d][4 * g + e] * inv);
                *reinterpret_cast<bf16x4_t*>(op + 32 * d + 8 * g + 4 * hw) = w;
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

}  // namespace

hipError_t launch_attn_bf16(const AttnArgs& a, int head_dim, hipStream_t s) {
    const dim3 grid(a.n_qtiles * a.B * a.H), block(kBf16Threads);
    if (head_dim == 128) {
        if (a.v_blocked) hipLaunchKernelGGL((attn_fwd_bf16_kernel<128, true>), grid, block, 0, s, a);
        else hipLaunchKernelGGL((attn_fwd_bf16_kernel<128, false>), grid, block, 0, s, a);
    } else if (head_dim == 64) {
        if (a.v_blocked) hipLaunchKernelGGL((attn_fwd_bf16_kernel<64, true>), grid, block, 0, s, a);
        else hipLaunchKernelGGL((attn_fwd_bf16_kernel<64, false>), grid, block, 0, s, a);
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
