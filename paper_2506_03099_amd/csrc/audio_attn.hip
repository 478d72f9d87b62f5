// Audio cross-attention with a local frame window and a face mask, for gfx950.
//
// TalkingMachines, Sec. 4.1: the DiT's cross-attention layers gain keys and
// values computed from audio tokens, which the tokens of each latent frame
// attend to; a local mask limits that attention to the face region; each
// latent frame sees only the audio tokens of the five latent frames centred
// on it; with several faces each face takes its own audio stream (a silent
// face's stream carries a special embedding, which is data to this kernel).
//
// Query row i (token of latent frame f = first_frame + i / T) with face id m
// in [0, M) attends to audio tokens [A * max(0, f - w), A * (min(F_a - 1,
// f + w) + 1)) of stream m: o_i = softmax(scale * q_i K^T) V, exact. Rows
// with face id -1 (or any id outside [0, M)) get zeros.
//
// Two kinds of workgroup share one launch:
//   - compute workgroups, one per (batch, head, latent frame, part of the
//     frame's 32-row blocks; a part takes every parts-th block), 8 waves:
//     waves 4-7 read the part's face ids into registers; then waves 0-3 issue
//     the direct global->LDS loads of stream 0's audio window (K and V rows,
//     16-byte chunks swizzled per row), before the face ids are known. Per
//     stream used by the part's rows, waves 4-7 compact the rows of that
//     stream into a list in row order (ballots, per-wave counts in LDS, one
//     prefix); every wave takes one dense 32-row block of the list and, once
//     the window has landed, computes it: S^T = K Q^T and O^T += V^T P^T with
//     v_mfma_f32_32x32x16_bf16 over groups of five 32-key tiles (the scores
//     of a group's tiles as independent MFMA chains, then the group's exact
//     row maximum, then P and the P V MFMAs tile by tile; O is rescaled only
//     when a later group raises some row's maximum), P kept in registers and
//     the V^T operand read with transposing LDS reads (ds_read_b64_tr_b16).
//     P is rounded to bf16 for the P V product; the row sums add the fp32 P.
//     The maximum is exact: the largest P of a row is then 1, which bf16
//     holds exactly, and over a window of a few hundred keys its weight
//     matters;
//   - zero-fill workgroups after them, each over a run of whole token rows
//     (all heads, contiguous in o): zeros for the rows without a face.
// Compacting the rows means the MFMAs run on dense blocks of face rows, not on
// every 32-row block that holds one. A dense block's 32 query rows are
// scattered in q, and so are its output rows: loaded or stored by the lanes
// that own them in the MFMA layout, every wave instruction touches 32 rows
// (32 cache lines) for 16 or 8 bytes each, and the vector memory unit spends
// its time on cache lines rather than bytes. Where LDS allows (a slot of 32
// rows per wave beside the window), the queries arrive by direct loads of
// whole rows (4 rows per instruction) into the wave's slot, in the K tiles'
// swizzled layout, and the bf16 output goes the same way back. The zero
// stores, most of the output, come from workgroups of their own: on this
// target a wait for a load also waits for the wave's earlier stores, and a
// CU's loads queue behind the stores it has issued, so zeros written by the
// compute workgroups would delay the loads on the critical path (face ids,
// queries). Every workgroup of the launch requests the same LDS, so at the
// usual window sizes a CU holds one of them and the zero-fill workgroups run
// on the CUs the compute workgroups leave free.
//
// The window is short (five frames of audio tokens), so the kernel is bound
// by memory traffic and latency, not by the MFMAs.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <atomic>

#include "tm_device.h"
#include "tm_internal.h"

namespace tmk {
namespace {

constexpr int kAudioThreads = 512;
constexpr int kAudioWaves = kAudioThreads / 64;

typedef __attribute__((address_space(3))) bf16x8_t lds_bf16x8_t;
typedef __attribute__((address_space(3))) bf16x4_t lds_bf16x4_t;
typedef __attribute__((address_space(3))) unsigned char lds_u8;
typedef __attribute__((address_space(3))) uint32_t lds_u32;
typedef __attribute__((address_space(3))) uint16_t lds_u16;
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) u32x4_t lds_u32x4_t;

// A lane value the compiler cannot see through: index math derived from it is
// computed where it is used, not hoisted ahead of a loop and kept live.
__device__ __forceinline__ int opaque(int v) {
    asm volatile("" : "+v"(v));
    return v;
}

// Workgroup barrier for LDS traffic: on gfx950 __syncthreads is
// s_waitcnt lgkmcnt(0) + s_barrier (its workgroup-scope fence needs no
// vector-memory wait), so this wave's LDS operations are complete while its
// global loads and stores may still be in flight.
__device__ __forceinline__ void lds_barrier() { __syncthreads(); }

// Zero-fill workgroup z: token rows [z * zrows, (z + 1) * zrows) of the
// B * n rows of o, every head (a whole row is H * D contiguous elements):
// zeros where the row's face id lies outside [0, M). Rows are taken in
// batches of at most 512, whose face flags are staged in LDS first.
template <int D, bool OF32>
__device__ __forceinline__ void zero_fill_rows(const AudioArgs& a, int z, lds_u8* flag) {
    constexpr int OES = OF32 ? 4 : 2;
    constexpr int ZB = 8;  // stores per pass whose flags are read together
    const int tid = threadIdx.x;
    const int64_t total = static_cast<int64_t>(a.B) * a.n;
    const int64_t r0 = static_cast<int64_t>(z) * a.zrows;
    const int64_t r1 = min(r0 + a.zrows, total);
    const int cpr = a.H * D * OES / 16;  // 16-byte chunks per token row (D * OES is a multiple of 16)
    // rows per batch: at most one per thread, and the batch's chunk count fits in 31 bits
    const int batch = max(1, min(kAudioThreads, 0x7fffffff / cpr));
    unsigned char* const ob = static_cast<unsigned char*>(a.o);
    for (int64_t rb = r0; rb < r1; rb += batch) {
        const int nr = static_cast<int>(min(static_cast<int64_t>(batch), r1 - rb));
        if (rb != r0) lds_barrier();  // every wave is done with the previous batch's flags
        if (tid < nr) {
            const int fid = a.face[rb + tid];
            flag[tid] = (fid >= 0 && fid < a.M) ? 1 : 0;  // 1: a face row, computed elsewhere
        }
        lds_barrier();
        const int n_chunks = nr * cpr;
        unsigned char* const base = ob + rb * cpr * 16;
        for (int i0 = tid; i0 < n_chunks; i0 += ZB * kAudioThreads) {
            unsigned char fz[ZB];
#pragma unroll
            for (int u = 0; u < ZB; ++u) fz[u] = flag[min(i0 + u * kAudioThreads, n_chunks - 1) / cpr];
#pragma unroll
            for (int u = 0; u < ZB; ++u) {
                const int i = i0 + u * kAudioThreads;
                if (i < n_chunks && fz[u] == 0)
                    store16_through(base + static_cast<int64_t>(i) * 16, u32x4_t{0, 0, 0, 0});
            }
        }
    }
}

template <int D, bool OF32, bool QS>
__global__ __launch_bounds__(kAudioThreads) void audio_attn_bf16_kernel(const AudioArgs a) {
    extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
    if (static_cast<int>(blockIdx.x) >= a.n_cwg) {  // uniform over the workgroup
        zero_fill_rows<D, OF32>(a, static_cast<int>(blockIdx.x) - a.n_cwg, (lds_u8*)(lds));
        return;
    }
    constexpr int ROWB = D * 2;   // bytes of a K or V row
    constexpr int CPR = D / 8;    // 16-byte chunks per row
    constexpr int KK = D / 16;    // k-steps of the score MFMA
    constexpr int DB = D / 32;    // 32-dimension blocks of the output
    constexpr int NCW = 4;        // waves 0..NCW-1 load the windows
    constexpr int NFW = 4;        // waves kAudioWaves-NFW.. read the face ids and compact
    constexpr int FT = NFW * 64;  // threads of the face waves
    constexpr int FID = 32 * kAudioBlocksPerPart / FT;  // face ids per face-wave thread
    static_assert(FID * FT == 32 * kAudioBlocksPerPart, "face ids must tile the face waves");
    static_assert(4 * (kAudioWaves + FID * NFW + 4) + 2 * 32 * kAudioBlocksPerPart == kAudioFaceLds,
                  "the LDS carve-up below must match kAudioFaceLds");

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l32 = lane & 31, hw = lane >> 5;
    const bool dma_wave = wave < NCW;
    const bool face_wave = wave >= kAudioWaves - NFW;
    const int fw = wave - (kAudioWaves - NFW);  // face wave index (valid for face waves)

    const int id = xcd_logical_id(blockIdx.x, a.n_cwg);
    const int part = id % a.parts;
    int rest = id / a.parts;
    const int fi = rest % a.n_frames;
    rest /= a.n_frames;
    const int h = rest % a.H;
    const int b = rest / a.H;

    // Rows of this workgroup: the frame's 32-row blocks part, part + parts,
    // ...; row i of the part (i = 32 j + r) is token row part_row(i).
    const int r_begin = fi * a.T;
    const int r_end = min(r_begin + a.T, a.n);
    const int nblk = (r_end - r_begin + 31) / 32;
    const int my_blk = nblk > part ? (nblk - part + a.parts - 1) / a.parts : 0;
    const int n_rows = 32 * my_blk;
    auto part_row = [&](int i) { return r_begin + 32 * (part + (i / 32) * a.parts) + i % 32; };

    // The frame's audio window.
    const int f = a.first_frame + fi;
    const int Fa = a.La / a.A;
    const int wlo = max(0, f - a.half_window), whi = min(Fa - 1, f + a.half_window);
    const int k_lo = wlo * a.A;
    const int nk = (whi - wlo + 1) * a.A;
    const int nk_pad = (nk + 31) & ~31;
    lds_u8* const Ks = (lds_u8*)(lds);
    lds_u8* const Vs = Ks + nk_pad * ROWB;
    // after the K and V areas of the launch's widest window: one word per wave
    // (streams used), the face waves' per-segment counts, the count of the
    // current stream's rows, those rows compacted (part-row indices) and, when
    // the queries are staged, one 32-row slot per wave
    lds_u32* const used_l = (lds_u32*)((lds_u8*)(lds) + 2 * a.max_keys_pad * ROWB);
    lds_u32* const cnt_l = used_l + kAudioWaves;
    lds_u32* const nf_l = cnt_l + FID * NFW;
    lds_u16* const list_l = (lds_u16*)(nf_l + 4);
    lds_u8* const slot = (lds_u8*)(list_l + 32 * kAudioBlocksPerPart) + wave * 32 * ROWB;

    const int64_t st = static_cast<int64_t>(a.H) * D;  // elements per token row
    const __bf16* qb = static_cast<const __bf16*>(a.q) + static_cast<int64_t>(b) * a.n * st + h * D;
    constexpr int OES = OF32 ? 4 : 2;   // bytes per output element
    unsigned char* ob = static_cast<unsigned char*>(a.o) + (static_cast<int64_t>(b) * a.n * st + h * D) * OES;
    const int32_t* fb = a.face + static_cast<int64_t>(b) * a.n;

    // Window of stream m into LDS by direct global->LDS loads issued by the
    // DMA waves (K and V rows in the same swizzled layout, so one lane offset
    // serves both): wave instruction i writes LDS chunks [64 i, 64 i + 64) of
    // each area and a lane fetches the global chunk that belongs at its
    // position. Rows past the window repeat its last row (finite values whose
    // scores are masked and whose P is exactly zero).
    const uint32_t lds_k = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(Ks));
    const uint32_t lds_v = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(Vs));
    auto stage_dma = [&](int m) {
        const int64_t kv_off = ((static_cast<int64_t>(b) * a.M + m) * a.La + k_lo) * st + h * D;
        const void* kg = uniform_ptr(static_cast<const __bf16*>(a.ak) + kv_off);
        const void* vg = uniform_ptr(static_cast<const __bf16*>(a.av) + kv_off);
        const int n_instr = nk_pad * CPR / 64;  // nk_pad is a multiple of 32, CPR of 8
        for (int i = wave; i < n_instr; i += NCW) {
            const int c = 64 * i + lane;
            const int k = c / CPR, pos = c % CPR;
            const int gc = pos ^ tr_swizzle<D>(k);
            const uint32_t off = static_cast<uint32_t>((min(k, nk - 1) * st + gc * 8) * 2);
            const uint32_t l = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(64 * i * 16));
            lds_dma16x2(kg, off, lds_k + l, vg, off, lds_v + l);
        }
    };

    // ---- face ids of the part's rows: face-wave thread t holds part rows
    // t + FT g (g < FID), so segment g (rows [FT g, FT g + FT)) is spread
    // over the face waves in row order. They are issued before the window
    // loads, which queue behind them.
    int fm[FID];
    if (face_wave) {
        const int ft = tid - (kAudioThreads - FT);
#pragma unroll
        for (int g = 0; g < FID; ++g) {
            const int i = ft + g * FT;
            fm[g] = fb[min(part_row(min(i, max(n_rows - 1, 0))), a.n - 1)];
        }
    }
    lds_barrier();  // the face-id loads go out first
    // stream 0's window is the first one needed unless stream 0 is not used:
    // its loads go out before the face ids are known
    if (dma_wave) stage_dma(0);
    uint32_t used = 0;
    if (face_wave) {
        const int ft = tid - (kAudioThreads - FT);
#pragma unroll
        for (int g = 0; g < FID; ++g) {
            const int i = ft + g * FT;
            int fid = (fm[g] >= 0 && fm[g] < a.M) ? fm[g] : -1;
            if (i >= n_rows || part_row(i) >= r_end) fid = -2;  // -2: no row here
            fm[g] = fid;
            if (fid >= 0) used |= 1u << fid;
        }
        // streams used by the wave's rows
        uint32_t wused = 0;
        for (int m = 0; m < a.M; ++m)
            if (__ballot((used >> m) & 1u) != 0) wused |= 1u << m;
        used = wused;
    }
    if (lane == 0) used_l[wave] = used;
    lds_barrier();
    uint32_t streams = 0;
#pragma unroll
    for (int w = 0; w < kAudioWaves; ++w) streams |= used_l[w];

    const float c = a.scale_log2;
    // Per-lane LDS byte offsets of the operand fragments of a 32-key tile
    // starting at a multiple of 16 rows (the swizzle depends on row % 16).
    // K fragment kk: row l32, chunk 2*kk + hw. V^T fragment (step j, block d):
    // two transposing reads of the row-major V rows 16*j + 4*hw + gi/4 (and
    // + 8), element columns 32*d + 16*(grp & 1) + 4*(gi & 3); with these, the
    // S^T output register i of a lane holds key 8*(i/4) + 4*hw + i%4, and its
    // P^T element for step i/8, slot i%8, matches the V^T row order.
    uint32_t koff[KK];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) koff[kk] = l32 * ROWB + (((2 * kk + hw) ^ tr_swizzle<D>(l32)) << 4);
    const int grp = lane >> 4, gi = lane & 15;
    const int v_row = 4 * hw + (gi >> 2);
    const int v_cbase = 2 * (grp & 1) + ((gi & 3) >> 1);
    const int v_half = (gi & 1) * 8;
    uint32_t voff[2 * DB];
#pragma unroll
    for (int d = 0; d < DB; ++d) {
        const int cc = 4 * d + v_cbase;
        voff[2 * d] = v_row * ROWB + ((cc ^ tr_swizzle<D>(v_row)) << 4) + v_half;
        voff[2 * d + 1] = (v_row + 8) * ROWB + ((cc ^ tr_swizzle<D>(v_row + 8)) << 4) + v_half;
    }

    // Query fragments of row `row`: lane l32's row, the half-wave's k-slices.
    auto load_q = [&](bf16x8_t (&qf)[KK], int row) __attribute__((always_inline)) {
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
            qf[kk] = *reinterpret_cast<const bf16x8_t*>(qb + row * st + kk * 16 + hw * 8);
    };
    // The rows of dense block jb of the current stream's compacted list:
    // lane l32 takes entry 32 jb + l32 (past the count: the last entry, whose
    // result is not stored).
    auto dense_row = [&](int jb, int nf) {
        return part_row(static_cast<int>(list_l[min(32 * jb + l32, nf - 1)]));
    };
    // Staged form: the 32 query rows of dense block jb into the wave's slot by
    // direct global->LDS loads of whole rows (4 rows per wave instruction, in
    // the K tiles' swizzled layout), so that a fragment read is koff[kk] into
    // the slot. A lane fetches the global chunk that belongs at its position.
    const uint32_t lds_slot = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(slot));
    auto stage_q = [&](int jb, int nf) __attribute__((always_inline)) {
        const void* qs = uniform_ptr(qb);
#pragma unroll
        for (int i = 0; i < 32 * CPR / 64; ++i) {
            const int cidx = 64 * i + lane;
            const int r = cidx / CPR, pos = cidx % CPR;
            const int gc = pos ^ tr_swizzle<D>(r);
            const int tok = part_row(static_cast<int>(list_l[min(32 * jb + r, nf - 1)]));
            const uint32_t off = static_cast<uint32_t>((tok * st + gc * 8) * 2);
            lds_dma16(qs, off, static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(lds_slot + 64 * i * 16)));
        }
    };

    // One dense block: S^T = K Q^T and O^T += V^T P^T over the window's
    // 32-key tiles, taken in groups of kGroup tiles (one group for a window
    // of five frames of 32 audio tokens). Per group: the scores of all its
    // tiles (independent MFMA chains, so the matrix core never waits for a
    // result), the group's exact row maximum (O and the row sums rescaled
    // when a later group raises it), then tile by tile P and its P V MFMAs.
    // Tiles of the last group past the window's end score a copy of its last
    // tile, are masked out and skip P V. O is stored for the lanes that hold
    // one of the stream's rows.
    constexpr int kGroup = 5;
    auto do_block = [&](int jb, int nf, const bf16x8_t (&qf)[KK]) __attribute__((always_inline)) {
        constexpr int NF = KK * kGroup;  // score MFMAs of a group
        constexpr int RING = 4;          // K fragments read ahead of their MFMA
        const int row = dense_row(jb, nf);
        const bool act = 32 * jb + l32 < nf;
        f32x16_t acc[DB];
#pragma unroll
        for (int d = 0; d < DB; ++d) acc[d] = f32x16_t{};
        float m_run = 0.f, l_run = 0.f;
        const int ntile = nk_pad / 32;
        for (int g0 = 0; g0 < ntile; g0 += kGroup) {
            f32x16_t s[kGroup];
            // MFMA j takes k-step j / kGroup of tile g0 + j % kGroup
            auto kfrag = [&](int j) __attribute__((always_inline)) {
                const int t = min(g0 + j % kGroup, ntile - 1);
                return *(lds_bf16x8_t*)(Ks + t * 32 * ROWB + koff[j / kGroup]);
            };
            bf16x8_t ring[RING];
#pragma unroll
            for (int j = 0; j < RING; ++j) ring[j] = kfrag(j);
            // staged queries: the fragment of k-step kk is read from the slot
            // one k-step ahead (two held), not kept for the whole block
            bf16x8_t qr[2];
            if constexpr (QS) qr[0] = *(lds_bf16x8_t*)(slot + koff[0]);
#pragma unroll
            for (int j = 0; j < NF; ++j) {
                const int u = j % kGroup, kk = j / kGroup;
                if constexpr (QS)
                    if (u == 0 && kk + 1 < KK) qr[(kk + 1) & 1] = *(lds_bf16x8_t*)(slot + koff[kk + 1]);
                const bf16x8_t qk = QS ? qr[kk & 1] : qf[kk];
                s[u] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ring[j % RING], qk, kk == 0 ? f32x16_t{} : s[u],
                                                               0, 0, 0);
                if (j + RING < NF) ring[j % RING] = kfrag(j + RING);
                __builtin_amdgcn_sched_barrier(0);
            }
            // keys past the window (its last tile, and tiles past it) never count
            if (32 * (g0 + kGroup) > nk) {
#pragma unroll
                for (int u = 0; u < kGroup; ++u)
#pragma unroll
                    for (int i = 0; i < 16; ++i)
                        if (32 * (g0 + u) + 8 * (i / 4) + 4 * hw + (i % 4) >= nk) s[u][i] = kNegInf;
            }
            float mx = s[0][0];
#pragma unroll
            for (int u = 0; u < kGroup; ++u)
#pragma unroll
                for (int i = (u == 0 ? 1 : 0); i < 16; i += 2)
                    mx = i + 1 < 16 ? fmaxf(mx, fmaxf(s[u][i], s[u][i + 1])) : fmaxf(mx, s[u][i]);
            const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx),
                                                             false, false);
            // every group holds a key of the window: the row's maximum is finite
            const float mt = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1])) * c;
            if (g0 == 0) {
                m_run = mt;
            } else if (__ballot(mt > m_run) != 0) {  // O rescaled only when some row's max rose
                const float m_new = fmaxf(m_run, mt);
                const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
                m_run = m_new;
                l_run *= alpha;
#pragma unroll
                for (int d = 0; d < DB; ++d) acc[d] *= alpha;
            }
            // P rounded to bf16 for the P V product; the row sums add the fp32
            // P. P of tile u + 1 is formed while the P V MFMAs of tile u run:
            // each of those MFMAs is followed by two of its elements (tiles
            // past the window give P = 0).
            float lsum = 0.f;
            auto p_pair = [&](int u, int i, bf16x8_t (&pn)[2]) __attribute__((always_inline)) {
                const float p0 = __builtin_amdgcn_exp2f(fmaf(s[u][i], c, -m_run));
                const float p1 = __builtin_amdgcn_exp2f(fmaf(s[u][i + 1], c, -m_run));
                pn[i / 8][i % 8] = static_cast<__bf16>(p0);
                pn[i / 8][i % 8 + 1] = static_cast<__bf16>(p1);
                lsum += p0 + p1;
            };
            bf16x8_t pf[2];
#pragma unroll
            for (int i = 0; i < 16; i += 2) p_pair(0, i, pf);
#pragma unroll
            for (int u = 0; u < kGroup; ++u) {
                if (g0 + u >= ntile) break;
                const uint32_t tile = (g0 + u) * 32 * ROWB;
                bf16x8_t pn[2];
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int jj = 0; jj < 2; ++jj) {
                    bf16x8_t vf[DB];
#pragma unroll
                    for (int d = 0; d < DB; ++d) {
                        const uint32_t rows = tile + 16 * jj * ROWB;
                        const bf16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
                            (lds_bf16x4_t*)(Vs + rows + voff[2 * d]));
                        const bf16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
                            (lds_bf16x4_t*)(Vs + rows + voff[2 * d + 1]));
                        vf[d] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
                    }
#pragma unroll
                    for (int d = 0; d < DB; ++d) {
                        acc[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[d], pf[jj], acc[d], 0, 0, 0);
                        if (u + 1 < kGroup) {
#pragma unroll
                            for (int q = 0; q < 4 / DB; ++q) p_pair(u + 1, 2 * ((jj * DB + d) * (4 / DB) + q), pn);
                        }
                        __builtin_amdgcn_sched_barrier(0);
                    }
                }
                if (u + 1 < kGroup) {
                    pf[0] = pn[0];
                    pf[1] = pn[1];
                }
            }
            l_run += lsum;
        }
        const auto lsw = __builtin_amdgcn_permlane32_swap(__float_as_uint(l_run), __float_as_uint(l_run),
                                                          false, false);
        const float inv = 1.f / (__uint_as_float(lsw[0]) + __uint_as_float(lsw[1]));  // both half-waves
        if constexpr (QS && !OF32) {
            {
                // bf16 rows through the wave's slot (the same swizzled layout),
                // then stored whole: 4 rows per wave instruction
                asm volatile("" ::: "memory");  // the fragment reads of the slot come first
                const int ln = opaque(lane);
                const int r32 = ln & 31, h2 = ln >> 5;
#pragma unroll
                for (int d = 0; d < DB; ++d) {
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        bf16x4_t w;
#pragma unroll
                        for (int e = 0; e < 4; ++e) w[e] = static_cast<__bf16>(acc[d][4 * g + e] * inv);
                        *(lds_bf16x4_t*)(slot + r32 * ROWB + (((4 * d + g) ^ tr_swizzle<D>(r32)) << 4) + h2 * 8) = w;
                    }
                }
                asm volatile("" ::: "memory");
#pragma unroll
                for (int i = 0; i < 32 * CPR / 64; ++i) {
                    const int cidx = 64 * i + ln;
                    const int r = cidx / CPR, pos = cidx % CPR;
                    const u32x4_t v = *(lds_u32x4_t*)(slot + cidx * 16);
                    if (32 * jb + r < nf) {
                        const int tok = part_row(static_cast<int>(list_l[32 * jb + r]));
                        store16_through(ob + tok * st * 2 + ((pos ^ tr_swizzle<D>(r)) << 4), v);
                    }
                }
                asm volatile("" ::: "memory");  // the slot is free once these reads are done
                return;
            }
        }
        if (act) {
            unsigned char* op = ob + (row * st) * OES;
#pragma unroll
            for (int d = 0; d < DB; ++d) {
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int e0 = 32 * d + 8 * g + 4 * hw;  // first of the lane's 4 dimensions
                    if constexpr (OF32) {
                        float4 w;
                        w.x = acc[d][4 * g + 0] * inv;
                        w.y = acc[d][4 * g + 1] * inv;
                        w.z = acc[d][4 * g + 2] * inv;
                        w.w = acc[d][4 * g + 3] * inv;
                        *reinterpret_cast<float4*>(op + e0 * 4) = w;
                    } else {
                        bf16x4_t w;
#pragma unroll
                        for (int e = 0; e < 4; ++e) w[e] = static_cast<__bf16>(acc[d][4 * g + e] * inv);
                        *reinterpret_cast<bf16x4_t*>(op + e0 * 2) = w;
                    }
                }
            }
        }
    };

    // ---- each stream used by the part's rows. Every wave passes the same
    // barriers.
    bool first = true;
    while (streams != 0) {
        const int m = __builtin_ctz(streams);
        streams &= streams - 1;
        if (!first) lds_barrier();  // every wave is done with the previous window and list
        if (dma_wave && (!first || m != 0)) {
            wait_lds_dma();  // an earlier window load must not land after this one
            stage_dma(m);
        }
        first = false;
        // the part's rows of stream m, compacted in row order: each face wave
        // counts its rows of every segment, then places them after the rows
        // of the earlier segments and of the earlier face waves in this one
        if (face_wave) {
#pragma unroll
            for (int g = 0; g < FID; ++g) {
                const uint64_t mask = __ballot(fm[g] == m);
                if (lane == 0) cnt_l[g * NFW + fw] = static_cast<uint32_t>(__popcll(mask));
            }
        }
        lds_barrier();  // the counts are complete
        if (face_wave) {
            uint32_t done = 0;  // rows of stream m in the segments before g
#pragma unroll
            for (int g = 0; g < FID; ++g) {
                uint32_t before = done, seg = 0;
#pragma unroll
                for (int w = 0; w < NFW; ++w) {
                    const uint32_t n = cnt_l[g * NFW + w];
                    before += w < fw ? n : 0;
                    seg += n;
                }
                const bool mine = fm[g] == m;
                const uint64_t mask = __ballot(mine);
                if (mine)
                    list_l[before + __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                                             __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0))] =
                        static_cast<uint16_t>(tid - (kAudioThreads - FT) + g * FT);
                done += seg;
            }
            if (fw == 0 && lane == 0) nf_l[0] = done;
        }
        lds_barrier();  // the list is complete
        const int nf = static_cast<int>(nf_l[0]);
        const int nb = (nf + 31) / 32;
        bf16x8_t qf[KK];
        if (wave < nb) {
            if constexpr (QS) stage_q(wave, nf);
            else load_q(qf, dense_row(wave, nf));
        }
        wait_lds_dma();  // this wave's window loads and queries
        lds_barrier();   // the window is in place
        for (int jb = wave; jb < nb; jb += kAudioWaves) {
            if constexpr (QS) {
                if (jb != wave) {
                    __builtin_amdgcn_s_waitcnt(kWaitLgkmcnt0);  // the slot's last reads are done
                    stage_q(jb, nf);
                    wait_lds_dma();
                }
            } else if (jb != wave) {
                load_q(qf, dense_row(jb, nf));
            }
            do_block(jb, nf, qf);
        }
    }
    // no window load may still be writing LDS when the workgroup ends (a part
    // whose rows use no stream never waits for the speculative one)
    if (dma_wave) wait_lds_dma();
}

// The kernel's dynamic-LDS limit is raised once per device (to the largest
// size, which covers every launch); concurrent first calls set the same value.
constexpr int kMaxDevices = 64;

template <int D, bool OF32, bool QS>
hipError_t launch(const AudioArgs& a, unsigned grid, size_t lds, hipStream_t s) {
    static std::atomic<bool> attr_set[kMaxDevices];
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    if (!attr_set[dev].load(std::memory_order_acquire)) {
        e = hipFuncSetAttribute(reinterpret_cast<const void*>(&audio_attn_bf16_kernel<D, OF32, QS>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(kAudioMaxLds));
        if (e != hipSuccess) return e;
        attr_set[dev].store(true, std::memory_order_release);
    }
    hipLaunchKernelGGL((audio_attn_bf16_kernel<D, OF32, QS>), dim3(grid), dim3(kAudioThreads), lds, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_audio_attn_bf16(const AudioArgs& args, int head_dim, hipStream_t s) {
    AudioArgs a = args;
    const int64_t n_cwg = static_cast<int64_t>(a.B) * a.H * a.n_frames * a.parts;
    if (n_cwg < 1 || n_cwg > INT32_MAX / 2) return hipErrorInvalidValue;
    // Zero-fill workgroups: the CUs the compute workgroups leave free (a
    // quarter of the chip at least), with at least 16 token rows each.
    static std::atomic<int> cu_count[kMaxDevices];
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    int cus = cu_count[dev].load(std::memory_order_relaxed);
    if (cus == 0) {
        e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
        if (e != hipSuccess) return e;
        if (cus < 1) return hipErrorInvalidValue;
        cu_count[dev].store(cus, std::memory_order_relaxed);
    }
    const int64_t rows = static_cast<int64_t>(a.B) * a.n;
    int64_t nz = n_cwg < cus ? std::max<int64_t>(cus - n_cwg, cus / 4) : cus / 4;
    nz = std::max<int64_t>(1, std::min(nz, (rows + 15) / 16));
    const int64_t zrows = (rows + nz - 1) / nz;
    if (zrows > INT32_MAX) return hipErrorInvalidValue;
    nz = (rows + zrows - 1) / zrows;
    a.n_cwg = static_cast<int32_t>(n_cwg);
    a.zrows = static_cast<int32_t>(zrows);
    size_t lds = audio_lds_bytes(head_dim, a.max_keys_pad);
    if (lds > kAudioMaxLds) return hipErrorInvalidValue;
    // Queries and output rows go through LDS when the per-wave slots fit next
    // to the window and every row of a batch element lies within 4 GiB of its
    // base (the direct loads take 32-bit offsets).
    const size_t staged = lds + audio_stage_lds_bytes(head_dim);
    a.q_stage = staged <= kAudioMaxLds &&
                static_cast<int64_t>(a.n) * a.H * head_dim * 2 <= static_cast<int64_t>(0xffffffff);
    if (a.q_stage) lds = staged;
    const unsigned g = static_cast<unsigned>(n_cwg + nz);
    if (a.q_stage) {
        if (head_dim == 128) return a.o_f32 ? launch<128, true, true>(a, g, lds, s) : launch<128, false, true>(a, g, lds, s);
        if (head_dim == 64) return a.o_f32 ? launch<64, true, true>(a, g, lds, s) : launch<64, false, true>(a, g, lds, s);
    } else {
        if (head_dim == 128) return a.o_f32 ? launch<128, true, false>(a, g, lds, s) : launch<128, false, false>(a, g, lds, s);
        if (head_dim == 64) return a.o_f32 ? launch<64, true, false>(a, g, lds, s) : launch<64, false, false>(a, g, lds, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace tmk
