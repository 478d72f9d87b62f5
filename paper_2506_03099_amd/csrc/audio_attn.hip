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
// region, which covers neighbouring blocks, is spread over the parts). The
// workgroup reads its rows' face ids into LDS; for each stream its rows use,
// it stages that stream's window of K and V in LDS once (row-major, 16-byte
// chunks swizzled per row), and every wave runs its blocks that hold rows of
// the stream: S^T = K Q^T and O^T += V^T P^T with v_mfma_f32_32x32x16_bf16,
// P kept in registers, the V^T operand read with transposing LDS reads
// (ds_read_b64_tr_b16), P rounded to bf16 and the row sums taken from the
// rounded P. The running maximum is exact (the largest P of a row is 1, which
// bf16 holds exactly; with a window of a few hundred keys its weight matters),
// and O is rescaled only in tiles where some row's maximum rose. Rows without
// a face are zero-filled right after the face ids are known, so that those
// writes overlap the staging and the MFMA work.
//
// The window is short (five frames of audio tokens), so the kernel is bound
// by memory traffic and latency, not by the MFMAs. The workgroup barriers
// wait for LDS operations only, and the loads are not followed by selects or
// joins (rows past an end repeat the last row), so that the compiler does not
// make a wave wait for all of its outstanding memory operations.

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

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l32 = lane & 31, hw = lane >> 5;

    const int total = a.B * a.H * a.n_frames * a.parts;
    const int id = xcd_logical_id(blockIdx.x, total);
    const int part = id % a.parts;
    int rest = id / a.parts;
    const int fi = rest % a.n_frames;
    rest /= a.n_frames;
    const int h = rest % a.H;
    const int b = rest / a.H;

    // Rows of this workgroup: the frame's 32-row blocks part, part + parts,
    // part + 2 * parts, ... (strided, so that a face region, which covers
    // neighbouring blocks, is spread over all the frame's workgroups).
    const int r_begin = fi * a.T;
    const int r_end = min(r_begin + a.T, a.n);
    const int nblk = (r_end - r_begin + 31) / 32;
    const int my_blk = nblk > part ? (nblk - part + a.parts - 1) / a.parts : 0;  // blocks of this part
    auto block_row0 = [&](int j) { return r_begin + 32 * (part + j * a.parts); };

    // The frame's audio window.
    const int f = a.first_frame + fi;
    const int Fa = a.La / a.A;
    const int wlo = max(0, f - a.half_window), whi = min(Fa - 1, f + a.half_window);
    const int k_lo = wlo * a.A;
    const int nk = (whi - wlo + 1) * a.A;
    const int nk_pad = (nk + 31) & ~31;
    lds_u8* const Ks = (lds_u8*)(lds);
    lds_u8* const Vs = Ks + nk_pad * ROWB;

    const int64_t st = static_cast<int64_t>(a.H) * D;  // elements per token row
    const __bf16* qb = static_cast<const __bf16*>(a.q) + static_cast<int64_t>(b) * a.n * st + h * D;
    // output rows: bf16, or fp32 with OF32 (the same values before rounding)
    constexpr int OES = OF32 ? 4 : 2;   // bytes per output element
    constexpr int OCPR = D * OES / 16;  // 16-byte chunks per output row
    unsigned char* ob = static_cast<unsigned char*>(a.o) + (static_cast<int64_t>(b) * a.n * st + h * D) * OES;
    const int32_t* fb = a.face + static_cast<int64_t>(b) * a.n;

    constexpr int FID = (32 * kAudioBlocksPerPart + kAudioThreads - 1) / kAudioThreads;  // per thread
    constexpr int SLOTS = (kAudioMaxKeys<D> * CPR + kAudioThreads - 1) / kAudioThreads;
    const int n_rows = 32 * my_blk;
    auto part_row = [&](int i) { return block_row0(i / 32) + i % 32; };
    // face ids of the part's rows, then one word per wave of the streams
    // they use, after the K and V areas of the largest window of the launch
    lds_u32* const face_l = (lds_u32*)((lds_u8*)(lds) + 2 * a.max_keys_pad * ROWB);
    lds_u32* const used_l = face_l + 32 * kAudioBlocksPerPart;

    // Window loads of stream m into registers (rows past the window repeat
    // its last row: finite values whose scores are masked and whose P is
    // exactly zero), and their stores into LDS.
    auto stage_load = [&](int m, u32x4_t (&kv)[SLOTS], u32x4_t (&vv)[SLOTS]) {
        const int64_t kv_off = ((static_cast<int64_t>(b) * a.M + m) * a.La + k_lo) * st + h * D;
        const __bf16* kg = static_cast<const __bf16*>(a.ak) + kv_off;
        const __bf16* vg = static_cast<const __bf16*>(a.av) + kv_off;
#pragma unroll
        for (int g = 0; g < SLOTS; ++g) {
            {
                const int i = tid + g * kAudioThreads;
                const int k = min(i / CPR, nk - 1), ch = i % CPR;
                kv[g] = *reinterpret_cast<const u32x4_t*>(kg + k * st + ch * 8);
                vv[g] = *reinterpret_cast<const u32x4_t*>(vg + k * st + ch * 8);
            }
        }
    };
    auto stage_store = [&](const u32x4_t (&kv)[SLOTS], const u32x4_t (&vv)[SLOTS]) {
#pragma unroll
        for (int g = 0; g < SLOTS; ++g) {
            const int i = tid + g * kAudioThreads;
            const int k = i / CPR, ch = i % CPR;
            if (k < nk_pad) {
                const int pos = k * ROWB + ((ch ^ lds_swizzle<D>(k)) << 4);
                *(lds_u32x4_t*)(Ks + pos) = kv[g];
                *(lds_u32x4_t*)(Vs + pos) = vv[g];
            }
        }
    };
    // Query fragments of block j: every lane loads its row (rows past the
    // frame read its last row). A lane whose row belongs to another stream or
    // to no face computes a result that is never stored; the max and the sums
    // it takes stay within its own query row.
    bf16x8_t qf[KK];
    auto load_q = [&](int j) {
        const int row = min(block_row0(j) + l32, r_end - 1);
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
            qf[kk] = *reinterpret_cast<const bf16x8_t*>(qb + row * st + kk * 16 + hw * 8);
    };

    // ---- face ids of the part's rows into LDS, and the streams they use
    int fm[FID];
#pragma unroll
    for (int g = 0; g < FID; ++g) {
        const int i = tid + g * kAudioThreads;
        const int r = min(part_row(min(i, max(n_rows - 1, 0))), a.n - 1);
        fm[g] = fb[r];
    }
    int q_blk = -1;  // block whose queries qf holds
    uint32_t used = 0;
#pragma unroll
    for (int g = 0; g < FID; ++g) {
        const int i = tid + g * kAudioThreads;
        int f = (fm[g] >= 0 && fm[g] < a.M) ? fm[g] : -1;
        if (i >= n_rows || part_row(i) >= r_end) f = -2;  // -2: no row here
        if (i < n_rows) face_l[i] = static_cast<uint32_t>(f);
        if (f >= 0) used |= 1u << f;
    }
#pragma unroll
    for (int sh = 1; sh < 64; sh *= 2) used |= __shfl_xor(used, sh);
    if (lane == 0) used_l[wave] = used;
    lds_barrier();
    uint32_t streams = 0;
#pragma unroll
    for (int w = 0; w < kAudioWaves; ++w) streams |= used_l[w];

    // ---- zeros for the rows without a face
    for (int i = tid; i < n_rows * OCPR; i += kAudioThreads) {
        const int ri = i / OCPR;
        if (static_cast<int>(face_l[ri]) == -1)
            *reinterpret_cast<u32x4_t*>(ob + (part_row(ri) * st) * OES + (i % OCPR) * 16) = u32x4_t{0, 0, 0, 0};
    }
    const float c = a.scale_log2;
    const bf16x2_t ones = {static_cast<__bf16>(1.f), static_cast<__bf16>(1.f)};
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

    // The next of this wave's blocks (j, j + 8, ...) that holds a row of
    // stream m, or my_blk.
    int m = 0;
    auto next_block = [&](int j) {
        for (; j < my_blk; j += kAudioWaves)
            if (__ballot(static_cast<int>(face_l[32 * j + l32]) == m) != 0) break;
        return j;
    };

    // The blocks of stream m (its window staged in LDS): each wave computes
    // its blocks that hold rows of the stream.
    auto compute_stream = [&]() {
        // ---- each wave: its blocks with rows of stream m
        int j = next_block(wave);
        if (j < my_blk && j != q_blk) {
            load_q(j);
            q_blk = j;
        }
        while (j < my_blk) {
            const int row = block_row0(j) + l32;
            const bool act = static_cast<int>(face_l[32 * j + l32]) == m;
            f32x16_t acc[DB];
#pragma unroll
            for (int d = 0; d < DB; ++d) acc[d] = f32x16_t{};
            float m_run = 0.f, l_run = 0.f;
            // K fragments of the next tile are read while the P V MFMAs run, V
            // fragments right after the score MFMAs: the reads land while the
            // MFMAs and the softmax run
            bf16x8_t kf[KK];
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) kf[kk] = *(lds_bf16x8_t*)(Ks + koff[kk]);
            for (int k0 = 0; k0 < nk_pad; k0 += 32) {
                const uint32_t tile = k0 * ROWB;
                f32x16_t s = f32x16_t{};
#pragma unroll
                for (int kk = 0; kk < KK; ++kk)
                    s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kk], qf[kk], s, 0, 0, 0);
                bf16x8_t vf[2][DB];
#pragma unroll
                for (int jj = 0; jj < 2; ++jj) {
#pragma unroll
                    for (int d = 0; d < DB; ++d) {
                        const uint32_t rows = tile + 16 * jj * ROWB;
                        const bf16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
                            (lds_bf16x4_t*)(Vs + rows + voff[2 * d]));
                        const bf16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
                            (lds_bf16x4_t*)(Vs + rows + voff[2 * d + 1]));
                        vf[jj][d] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
                    }
                }
                // keys past the window (last tile only) never count
                if (k0 + 32 > nk) {
#pragma unroll
                    for (int i = 0; i < 16; ++i)
                        if (k0 + 8 * (i / 4) + 4 * hw + (i % 4) >= nk) s[i] = kNegInf;
                }
                float mx = s[0];
#pragma unroll
                for (int i = 1; i < 16; ++i) mx = fmaxf(mx, s[i]);
                const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx),
                                                                 false, false);
                // every tile holds a key of the window: the row's tile maximum is finite
                const float mt = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1])) * c;
                if (k0 == 0) {
                    m_run = mt;
                } else if (__ballot(mt > m_run) != 0) {  // O rescaled only when some row's max rose
                    const float m_new = fmaxf(m_run, mt);
                    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
                    m_run = m_new;
                    l_run *= alpha;
#pragma unroll
                    for (int d = 0; d < DB; ++d) acc[d] *= alpha;
                }
                bf16x8_t pf[2];
#pragma unroll
                for (int i = 0; i < 16; i += 2) {
                    const float p0 = __builtin_amdgcn_exp2f(fmaf(s[i], c, -m_run));
                    const float p1 = __builtin_amdgcn_exp2f(fmaf(s[i + 1], c, -m_run));
                    pf[i / 8][i % 8] = static_cast<__bf16>(p0);
                    pf[i / 8][i % 8 + 1] = static_cast<__bf16>(p1);
                    const bf16x2_t pp = {pf[i / 8][i % 8], pf[i / 8][i % 8 + 1]};
                    l_run = __builtin_amdgcn_fdot2_f32_bf16(pp, ones, l_run, false);
                }
#pragma unroll
                for (int jj = 0; jj < 2; ++jj) {
#pragma unroll
                    for (int d = 0; d < DB; ++d)
                        acc[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[jj][d], pf[jj], acc[d], 0, 0, 0);
                }
                if (k0 + 32 < nk_pad) {
#pragma unroll
                    for (int kk = 0; kk < KK; ++kk) kf[kk] = *(lds_bf16x8_t*)(Ks + tile + 32 * ROWB + koff[kk]);
                }
            }
            // the next block's queries are loaded before this block's stores
            const int jn = next_block(j + kAudioWaves);
            if (jn < my_blk) {
                load_q(jn);
                q_blk = jn;
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
            j = jn;
        }
    };

    // Each stream used by the part's rows: its window staged once every wave
    // is done with the previous one, then its blocks.
    bool first = true;
    while (streams != 0) {
        m = __builtin_ctz(streams);
        streams &= streams - 1;
        u32x4_t kv[SLOTS], vv[SLOTS];
        stage_load(m, kv, vv);
        if (!first) lds_barrier();
        first = false;
        stage_store(kv, vv);
        lds_barrier();
        compute_stream();
    }
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
