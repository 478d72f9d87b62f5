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
// One workgroup of 8 waves per (batch, head, latent frame, part of the
// frame's 32-row blocks; a part takes every parts-th block, so that a face
// region, which covers neighbouring blocks, is spread over the parts). Waves
// 0-3 stage and compute, waves 4-7 read the face ids and zero-fill:
//   - waves 0-3 issue direct global->LDS loads of stream 0's audio window (K
//     and V rows, 16-byte chunks swizzled per row) at once, before the face
//     ids are known; waves 4-7 read the part's face ids into LDS;
//   - per stream used by the part's rows: wave 0 compacts the rows of that
//     stream into a list (ballot prefix counts), each of waves 0-3 loads the
//     queries of one dense 32-row block of the list (a gather of rows), and
//     once the window and those queries have landed, waves 4-7 zero-fill the
//     rows without a face (first stream only) while waves 0-3 compute their
//     dense blocks: S^T = K Q^T and O^T += V^T P^T with
//     v_mfma_f32_32x32x16_bf16, the score MFMAs of the next 32-key tile issued
//     before the softmax of the current one, P kept in registers and the V^T
//     operand read with transposing LDS reads (ds_read_b64_tr_b16). P is
//     rounded to bf16 for the P V product; the row sums add the fp32 P. The
//     running maximum is exact (the largest P of a row is 1, which bf16 holds
//     exactly; with a window of a few hundred keys its weight matters), and O
//     is rescaled only in tiles where some row's maximum rose.
// Compacting the rows means the MFMAs run on dense blocks of face rows, not on
// every 32-row block that holds one. Waves 4-7 issue no load after their zero
// stores, and the stores begin only after the loads the computation needs
// have landed: on this target a wait for a load also waits for every earlier
// store of the wave, and loads queued behind the zeros arrive late.
//
// The window is short (five frames of audio tokens), so the kernel is bound
// by memory traffic and latency, not by the MFMAs.

#include <hip/hip_runtime.h>
#include <stdint.h>

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

// Workgroup barrier for LDS traffic: on gfx950 __syncthreads is
// s_waitcnt lgkmcnt(0) + s_barrier (its workgroup-scope fence needs no
// vector-memory wait), so this wave's LDS operations are complete while its
// global loads and stores may still be in flight.
__device__ __forceinline__ void lds_barrier() { __syncthreads(); }

template <int D, bool OF32>
__global__ __launch_bounds__(kAudioThreads) void audio_attn_bf16_kernel(const AudioArgs a) {
    extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
    constexpr int ROWB = D * 2;   // bytes of a K or V row
    constexpr int CPR = D / 8;    // 16-byte chunks per row
    constexpr int KK = D / 16;    // k-steps of the score MFMA
    constexpr int DB = D / 32;    // 32-dimension blocks of the output
    constexpr int NCW = kAudioWaves / 2;  // waves 0..NCW-1 stage and compute, the others zero-fill

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l32 = lane & 31, hw = lane >> 5;
    const bool compute_wave = wave < NCW;

    const int total = a.B * a.H * a.n_frames * a.parts;
    const int id = xcd_logical_id(blockIdx.x, total);
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
    // after the K and V areas of the launch's widest window: the part's face
    // ids, one word per wave (streams used), the compacted rows of the
    // current stream (part-row indices) and their count
    lds_u32* const face_l = (lds_u32*)((lds_u8*)(lds) + 2 * a.max_keys_pad * ROWB);
    lds_u32* const used_l = face_l + 32 * kAudioBlocksPerPart;
    lds_u16* const list_l = (lds_u16*)(used_l + kAudioWaves);
    lds_u32* const nf_l = (lds_u32*)(list_l + 32 * kAudioBlocksPerPart);

    const int64_t st = static_cast<int64_t>(a.H) * D;  // elements per token row
    const __bf16* qb = static_cast<const __bf16*>(a.q) + static_cast<int64_t>(b) * a.n * st + h * D;
    constexpr int OES = OF32 ? 4 : 2;   // bytes per output element
    constexpr int OCPR = D * OES / 16;  // 16-byte chunks per output row
    unsigned char* ob = static_cast<unsigned char*>(a.o) + (static_cast<int64_t>(b) * a.n * st + h * D) * OES;
    const int32_t* fb = a.face + static_cast<int64_t>(b) * a.n;

    // Window of stream m into LDS by direct global->LDS loads issued by the
    // compute waves (K and V rows in the same swizzled layout, so one lane
    // offset serves both): wave instruction i writes LDS chunks [64 i, 64 i +
    // 64) of each area and a lane fetches the global chunk that belongs at its
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
            const int gc = pos ^ lds_swizzle<D>(k);
            const uint32_t off = static_cast<uint32_t>((min(k, nk - 1) * st + gc * 8) * 2);
            const uint32_t l = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(64 * i * 16));
            lds_dma16x2(kg, off, lds_k + l, vg, off, lds_v + l);
        }
    };

    // ---- stream 0's window is the first one needed unless stream 0 is not
    // used: its loads go out before the face ids are known
    if (compute_wave) stage_dma(0);

    // ---- face ids of the part's rows into LDS, and the streams they use
    // (read by the zero-fill waves, which have no window loads in flight)
    constexpr int ZT = kAudioThreads - NCW * 64;  // threads of the zero-fill waves
    constexpr int FID = (32 * kAudioBlocksPerPart + ZT - 1) / ZT;  // per thread
    uint32_t used = 0;
    if (!compute_wave) {
        const int zt = tid - NCW * 64;
        int fm[FID];
#pragma unroll
        for (int g = 0; g < FID; ++g) {
            const int i = zt + g * ZT;
            fm[g] = fb[min(part_row(min(i, max(n_rows - 1, 0))), a.n - 1)];
        }
#pragma unroll
        for (int g = 0; g < FID; ++g) {
            const int i = zt + g * ZT;
            int fid = (fm[g] >= 0 && fm[g] < a.M) ? fm[g] : -1;
            if (i >= n_rows || part_row(i) >= r_end) fid = -2;  // -2: no row here
            if (i < n_rows) face_l[i] = static_cast<uint32_t>(fid);
            if (fid >= 0) used |= 1u << fid;
        }
    }
#pragma unroll
    for (int sh = 1; sh < 64; sh *= 2) used |= __shfl_xor(used, sh);
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
    for (int kk = 0; kk < KK; ++kk) koff[kk] = l32 * ROWB + (((2 * kk + hw) ^ lds_swizzle<D>(l32)) << 4);
    const int grp = lane >> 4, gi = lane & 15;
    const int v_row = 4 * hw + (gi >> 2);
    const int v_cbase = 2 * (grp & 1) + ((gi & 3) >> 1);
    const int v_half = (gi & 1) * 8;
    uint32_t voff[2 * DB];
#pragma unroll
    for (int d = 0; d < DB; ++d) {
        const int cc = 4 * d + v_cbase;
        voff[2 * d] = v_row * ROWB + ((cc ^ lds_swizzle<D>(v_row)) << 4) + v_half;
        voff[2 * d + 1] = (v_row + 8) * ROWB + ((cc ^ lds_swizzle<D>(v_row + 8)) << 4) + v_half;
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

    // One dense block: S^T = K Q^T and O^T += V^T P^T over the window's
    // 32-key tiles with an exact running maximum; O stored for the lanes
    // that hold one of the stream's rows.
    auto do_block = [&](int jb, int nf, const bf16x8_t (&qf)[KK]) __attribute__((always_inline)) {
        const int row = dense_row(jb, nf);
        const bool act = 32 * jb + l32 < nf;
        f32x16_t acc[DB];
#pragma unroll
        for (int d = 0; d < DB; ++d) acc[d] = f32x16_t{};
        float m_run = 0.f, l_run = 0.f;
        // The score MFMAs of tile t+1 are issued before the softmax of tile t,
        // so that the matrix core works while the wave forms P; K fragments
        // are read one tile ahead of their MFMAs, V fragments right after the
        // score MFMAs.
        const int ntile = nk_pad / 32;
        bf16x8_t kf[KK];
        auto read_k = [&](int t) __attribute__((always_inline)) {
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) kf[kk] = *(lds_bf16x8_t*)(Ks + t * 32 * ROWB + koff[kk]);
        };
        auto scores = [&](f32x16_t& s) __attribute__((always_inline)) {
            s = f32x16_t{};
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kk], qf[kk], s, 0, 0, 0);
        };
        f32x16_t s_cur, s_nxt;
        read_k(0);
        scores(s_cur);
        if (ntile > 1) read_k(1);
        for (int t = 0; t < ntile; ++t) {
            const int k0 = 32 * t;
            const uint32_t tile = k0 * ROWB;
            if (t + 1 < ntile) {
                scores(s_nxt);
                if (t + 2 < ntile) read_k(t + 2);
            }
            f32x16_t s = s_cur;
            // keys past the window (last tile only) never count
            if (k0 + 32 > nk) {
#pragma unroll
                for (int i = 0; i < 16; ++i)
                    if (k0 + 8 * (i / 4) + 4 * hw + (i % 4) >= nk) s[i] = kNegInf;
            }
            float mx = fmaxf(fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3])), fmaxf(fmaxf(s[4], s[5]), fmaxf(s[6], s[7])));
            mx = fmaxf(mx, fmaxf(fmaxf(fmaxf(s[8], s[9]), fmaxf(s[10], s[11])),
                                 fmaxf(fmaxf(s[12], s[13]), fmaxf(s[14], s[15]))));
            const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx),
                                                             false, false);
            // every tile holds a key of the window: the row's tile maximum is finite
            const float mt = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1])) * c;
            if (t == 0) {
                m_run = mt;
            } else if (__ballot(mt > m_run) != 0) {  // O rescaled only when some row's max rose
                const float m_new = fmaxf(m_run, mt);
                const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
                m_run = m_new;
                l_run *= alpha;
#pragma unroll
                for (int d = 0; d < DB; ++d) acc[d] *= alpha;
            }
            // P rounded to bf16 for the P V product; the row sums add the fp32 P
            bf16x8_t pf[2];
            float l0 = 0.f, l1 = 0.f;
#pragma unroll
            for (int i = 0; i < 16; i += 2) {
                const float p0 = __builtin_amdgcn_exp2f(fmaf(s[i], c, -m_run));
                const float p1 = __builtin_amdgcn_exp2f(fmaf(s[i + 1], c, -m_run));
                pf[i / 8][i % 8] = static_cast<__bf16>(p0);
                pf[i / 8][i % 8 + 1] = static_cast<__bf16>(p1);
                l0 += p0;
                l1 += p1;
            }
            l_run += l0 + l1;
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
                for (int d = 0; d < DB; ++d)
                    acc[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[d], pf[jj], acc[d], 0, 0, 0);
            }
            s_cur = s_nxt;
        }
        const auto lsw = __builtin_amdgcn_permlane32_swap(__float_as_uint(l_run), __float_as_uint(l_run),
                                                          false, false);
        const float inv = 1.f / (__uint_as_float(lsw[0]) + __uint_as_float(lsw[1]));  // both half-waves
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
    // barriers; only the compute waves stage, compact and compute.
    bool first = true;
    const int first_m = streams != 0 ? __builtin_ctz(streams) : -1;
    while (streams != 0) {
        const int m = __builtin_ctz(streams);
        streams &= streams - 1;
        if (!first) lds_barrier();  // every wave is done with the previous window and list
        if (compute_wave) {
            if (!first || m != 0) {
                wait_lds_dma();  // an earlier window load must not land after this one
                stage_dma(m);
            }
            // wave 0: the part's rows of stream m, compacted in row order
            if (wave == 0) {
                int nf = 0;
                for (int c0 = 0; c0 < n_rows; c0 += 64) {
                    const bool mine = c0 + lane < n_rows && static_cast<int>(face_l[c0 + lane]) == m;
                    const uint64_t mask = __ballot(mine);
                    if (mine) list_l[nf + __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                       __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0))] =
                        static_cast<uint16_t>(c0 + lane);
                    nf += __popcll(mask);
                }
                if (lane == 0) nf_l[0] = static_cast<uint32_t>(nf);
            }
        }
        first = false;
        lds_barrier();  // the list is complete
        const int nf = static_cast<int>(nf_l[0]);
        const int nb = (nf + 31) / 32;
        bf16x8_t qf[KK];
        if (compute_wave) {
            if (wave < nb) load_q(qf, dense_row(wave, nf));
            wait_lds_dma();  // this wave's window loads and queries
        }
        lds_barrier();  // the window is in place
        // zero-fill waves, once, after the first window and the compute
        // waves' queries have landed (issued earlier, these loads would wait
        // behind the zeros): zeros for the rows without a face. They issue no
        // load afterwards (a wait for a load would also wait for these stores).
        if (!compute_wave && m == first_m) {
            // 16-byte chunk i of the part's output rows (OCPR per row); the face
            // ids of ZB consecutive iterations are read before their stores
            constexpr int ZS = kAudioThreads - NCW * 64;
            constexpr int ZB = 8;
            const int n_chunks = n_rows * OCPR;
            for (int i0 = tid - NCW * 64; i0 < n_chunks; i0 += ZB * ZS) {
                int fz[ZB];
#pragma unroll
                for (int u = 0; u < ZB; ++u) fz[u] = static_cast<int>(face_l[min(i0 + u * ZS, n_chunks - 1) / OCPR]);
#pragma unroll
                for (int u = 0; u < ZB; ++u) {
                    const int i = i0 + u * ZS;
                    if (i < n_chunks && fz[u] == -1)
                        *reinterpret_cast<u32x4_t*>(ob + (part_row(i / OCPR) * st) * OES + (i % OCPR) * 16) =
                            u32x4_t{0, 0, 0, 0};
                }
            }
        }
        if (compute_wave) {
            for (int jb = wave; jb < nb; jb += NCW) {
                if (jb != wave) load_q(qf, dense_row(jb, nf));
                do_block(jb, nf, qf);
            }
        }
    }
    // no window load may still be writing LDS when the workgroup ends (a part
    // whose rows use no stream never waits for the speculative one)
    if (compute_wave) wait_lds_dma();
}

// The kernel's dynamic-LDS limit is raised once per device (to the largest
// size, which covers every launch); concurrent first calls set the same value.
constexpr int kMaxDevices = 64;

template <int D, bool OF32>
hipError_t launch(const AudioArgs& a, unsigned grid, size_t lds, hipStream_t s) {
    static std::atomic<bool> attr_set[kMaxDevices];
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    if (!attr_set[dev].load(std::memory_order_acquire)) {
        e = hipFuncSetAttribute(reinterpret_cast<const void*>(&audio_attn_bf16_kernel<D, OF32>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(kAudioMaxLds));
        if (e != hipSuccess) return e;
        attr_set[dev].store(true, std::memory_order_release);
    }
    hipLaunchKernelGGL((audio_attn_bf16_kernel<D, OF32>), dim3(grid), dim3(kAudioThreads), lds, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_audio_attn_bf16(const AudioArgs& a, int head_dim, hipStream_t s) {
    const int64_t grid = static_cast<int64_t>(a.B) * a.H * a.n_frames * a.parts;
    if (grid < 1 || grid > INT32_MAX) return hipErrorInvalidValue;
    const size_t lds = audio_lds_bytes(head_dim, a.max_keys_pad);
    if (lds > kAudioMaxLds) return hipErrorInvalidValue;
    const unsigned g = static_cast<unsigned>(grid);
    if (head_dim == 128) return a.o_f32 ? launch<128, true>(a, g, lds, s) : launch<128, false>(a, g, lds, s);
    if (head_dim == 64) return a.o_f32 ? launch<64, true>(a, g, lds, s) : launch<64, false>(a, g, lds, s);
    return hipErrorInvalidValue;
}

}  // namespace tmk
