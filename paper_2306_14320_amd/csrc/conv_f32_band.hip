// fp32 im2win convolution by bands of output rows: a workgroup computes a
// band of rows of one image (or, for feature maps smaller than a band,
// several whole images) for 32 or 64 output channels, with every SIMD
// busy on the same amount of matrix-core work (one wave each, or two for the
// two-way split), so that a layer of a few hundred workgroups fills the chip
// without the quantization of fixed pixel tiles.
//
// The same implicit GEMM as the other convolution kernels (Alg. 2: the
// window of output pixel (m, n) is the run [n*sw*Fh, (n*sw + Fw)*Fh) of
// window-tensor row m; tap (u, v) sits at offset v*Fh + u):
//   - the band's NB blocks of 32 pixels each meet one block of 32 output
//     channels in v_mfma_f32_32x32x2f32 (A = 32 filter rows, B = 32 pixel
//     windows);
//   - the reduction runs over chunks of 8 input channels, 4 pairs (one
//     channel per k-slot of the matrix core).  With KS = 4 the waves take one
//     pair each for 32 output channels; with KS = 2 they split into 2 blocks
//     of 32 output channels x 2 halves of the pairs.  The partial sums of a
//     block's KS waves are added in a fixed order through LDS at the end;
//   - a chunk's strips (the band's window-tensor rows, one slot per channel,
//     in the window tensor's own layout) sit in LDS two chunks deep.
//     Unfused, each channel's strip is one contiguous run of the window
//     tensor, copied by LDS DMA (buffer_load ... lds, no register round
//     trip) in 16-byte pieces, or 4-byte ones when the planes are not
//     16-byte aligned.  Fused, the slot holds the band's input rows instead
//     (raw mode), each with zero columns on both sides, copied in 16-byte
//     pieces several rows per copy: the window of pixel (m, n) then starts at
//     raw row (m - m0)*sh, column n*sw - pw, and tap (u, v) lies u rows and
//     v columns further, a fixed offset as in the window tensor.  Where the
//     input rows are not whole 16-byte vectors, every strip element is
//     gathered from x by 4-byte LDS DMA instead.  Per-lane source offsets
//     are computed once per kernel; padding positions carry an offset past
//     the end of the buffer, which the hardware reads as zero;
//   - the filter does not go through LDS: each lane loads its own filter
//     rows (one output channel, one input channel per pair, Fh*Fw taps) of
//     the next chunk into registers while the current chunk is multiplied;
//   - the copies of the next chunk are spread over the taps of the current
//     one, and the windows of the next tap are read before the MFMAs of the
//     current tap, so both latencies hide behind matrix-core work.
// Both variants multiply the same values in the same matrix-core sequence,
// so their outputs are bitwise identical.
// Consecutive workgroups (the output-channel groups and bands of one image)
// are placed on the same XCD (the hardware hands consecutive workgroup ids
// to the 8 XCDs in turn), so they share the image in that XCD's L2.
#include "conv_common.h"

#include <cstdio>
#include <type_traits>

namespace im2win {
namespace {

typedef __attribute__((address_space(3))) void lds_void;

// Raw buffer resource over `bytes` bytes at p (loads past the end read 0).
__device__ inline __amdgpu_buffer_rsrc_t band_rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

// Element r of a vector, by value (a bit cast of the element expression
// itself compiles to element 0).
__device__ inline float elem(const f32x16& v, int r) { return v[r]; }

// Scheduling fence that keeps global/buffer memory accesses where they are
// issued while LDS reads and MFMAs may still interleave across it.
#define BAND_PIN_VMEM() __builtin_amdgcn_sched_barrier(0x0001 | 0x0002 | 0x0004 | 0x0008 | 0x0080 | 0x0100 | 0x0200)

template <int FH, int FW, int NB, int MODE, int KS>
__global__ __launch_bounds__(kBandThreads, 1) void conv_f32_band_kernel(F32BandArgs a) {
    constexpr int T = FH * FW;
    constexpr int PP = 4 / KS;                       // channel pairs of a chunk per wave
    constexpr int CB = 4 / KS;                       // blocks of 32 output channels per workgroup
    constexpr int STEPS = PP * T;                    // k-steps of a chunk per wave
    constexpr int NJ = band_copies(MODE);            // copies per wave per chunk
    constexpr int NS = NJ / 2;                       // copies per channel slot
    constexpr int DPT = (NJ + STEPS - 1) / STEPS;    // copies issued after each k-step
    constexpr int PAIR_B = 2 * kBandSlot * 4;        // LDS bytes from one pair's slots to the next
    extern __shared__ __align__(16) float S[];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform (scalar registers)
    const int cb = wv / KS, ks = wv - cb * KS;      // output-channel block, share of the pairs
    const int bid = a.xcd_remap ? (int)(blockIdx.x & 7) * (a.grid >> 3) + (int)(blockIdx.x >> 3)
                                : (int)blockIdx.x;
    const BandTile tile = band_tile(a, bid);
    const int slot = lane >> 5;     // k-slot: channel 2*p + slot of pair p
    const int col = lane & 31;      // A: output channel; B: pixel b*32 + col
    const int kout = (tile.kt * CB + cb) * 32 + col;

    // Window start (LDS byte address, stage 0, first pair of this wave) of
    // the lane's pixel in each pixel block.  The stage, the pair and the tap
    // are immediate offsets of the read.
    uint32_t bb[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) bb[b] = band_window(a, tile, FH, 2 * ks * PP + slot, lane, b);

    // Filter rows of this lane: output channel kout, input channel
    // ch*8 + 2*(ks*PP + pp) + slot for pair pp, taps 0 .. T-1 (natural (u, v)
    // order).
    const __amdgpu_buffer_rsrc_t wres = band_rsrc(a.wt, (uint32_t)((size_t)a.k * a.c * T * 4));
    const int wlane = ((kout * a.c) + 2 * ks * PP + slot) * T * 4;

    // Source of the staging copies: the image's window-tensor planes, or the
    // image's input planes.
    const size_t img_elems = (size_t)a.c * a.plane_src;
    const __amdgpu_buffer_rsrc_t sres =
        band_rsrc(a.src + (size_t)tile.img * img_elems, (uint32_t)(tile.nimg * img_elems * 4));
    const int plane_bytes = a.plane_src * 4;

    // Per-lane source byte offset (within one channel plane) of each copy of
    // a slot, the same for every channel and chunk (band_source).  Copies
    // past the strip or into the padding read from outside the buffer, which
    // yields zeros, so every copy is issued unconditionally and the slot's
    // tail beyond the strip is never read.
    uint32_t sofs[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) sofs[s] = band_source(a, tile, MODE, FH, s, lane);

    // Copy j of chunk ch into stage ST: channel slot 2*wv + (j & 1), part
    // j >> 1.  A chunk past the last one reads only zeros (harmless: that
    // stage is not read again).
    // Raw mode: copies past the band's rgroups are skipped, and so are the
    // lanes past rrpi whole rows.
    auto copy = [&](int j, int ch, auto st_tag) {
        constexpr int ST = decltype(st_tag)::value;
        if (MODE == kBandRaw && (j >> 1) >= a.rgroups) return;
        const uint32_t cbytes = (uint32_t)((ch * kBandChunk + 2 * wv + (j & 1)) * plane_bytes);
        char* dst = reinterpret_cast<char*>(S) + ST * kBandStageBytes + band_dest(a, MODE, wv, j);
        if (MODE != kBandRaw || lane < a.rrpi * a.rlanes) {
#if defined(__HIP_DEVICE_COMPILE__)   // (16-byte LDS copies exist on gfx950 only; the host pass checks them too)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(sres, (lds_void*)dst,
                                                     MODE == kBandWide || MODE == kBandRaw ? 16 : 4,
                                                     sofs[j >> 1] + cbytes, 0, 0, 0);
#endif
        }
    };

    float fa0[STEPS], fa1[STEPS];
    auto load_filter = [&](int ch, int q) {   // k-step q = pp*T + t
        const int pp = q / T, t = q - pp * T;
        return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                             wres, wlane + (2 * pp * T + t) * 4, ch * kBandChunk * T * 4, 0));
    };

    f32x16 acc[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[b][r] = 0.0f;

    // One chunk from stage ST with filter registers fa, while the copies of
    // chunk ch + 1 into the other stage and its filter rows (into fn) are
    // issued between the k-steps.  The windows of step q + 1 are read before
    // the MFMAs of step q; the scheduling fences keep the reads ahead of the
    // copies, which the compiler cannot tell apart from the stage being read.
    auto chunk = [&](auto st_tag, const float (&fa)[STEPS], float (&fn)[STEPS], int ch) {
        constexpr int ST = decltype(st_tag)::value;
        const char* base = reinterpret_cast<const char*>(S) + ST * kBandStageBytes;
        float bv[2][NB];
        auto read_step = [&](int q, float (&dst)[NB]) {
            const int pp = q / T, t = q - pp * T;
            const int u = t / FW, v = t - u * FW;
            const int off = pp * PAIR_B + (MODE == kBandRaw ? (u * a.rpitch + v) * 4 : (v * FH + u) * 4);
#pragma unroll
            for (int b = 0; b < NB; ++b) dst[b] = *reinterpret_cast<const float*>(base + bb[b] + off);
        };
        read_step(0, bv[0]);
#pragma unroll
        for (int q = 0; q < STEPS; ++q) {
            if (q + 1 < STEPS) read_step(q + 1, bv[(q + 1) & 1]);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int b = 0; b < NB; ++b)
                acc[b] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[q], bv[q & 1][b], acc[b], 0, 0, 0);
            BAND_PIN_VMEM();
#pragma unroll
            for (int d = 0; d < DPT; ++d)
                if (q * DPT + d < NJ) copy(q * DPT + d, ch + 1, std::integral_constant<int, 1 - ST>());
            fn[q] = load_filter(ch + 1, q);
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    // Waits for this wave's copies and filter loads (vector-memory counter
    // 0; the other counters at their maximum), then for the other waves.
    auto land = [&]() {
        __builtin_amdgcn_s_waitcnt(0x0F70);
        __syncthreads();
    };

#pragma unroll
    for (int j = 0; j < NJ; ++j) copy(j, 0, std::integral_constant<int, 0>());
#pragma unroll
    for (int q = 0; q < STEPS; ++q) fa0[q] = load_filter(0, q);
    land();
    for (int ch = 0; ch < a.nchunks; ch += 2) {   // nchunks is even
        chunk(std::integral_constant<int, 0>(), fa0, fa1, ch);
        land();
        chunk(std::integral_constant<int, 1>(), fa1, fa0, ch + 1);
        land();
    }

    constexpr int RP = NB * 32;
    constexpr int RW = 32 * RP;   // floats per partial
    if constexpr (KS == 4) {
        // All four partial sums go to LDS (R[wave][channel][pixel]); every
        // thread then adds one pixel's four partials in order,
        // ((P0 + P1) + P2) + P3, for all 32 channels.
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int ch = (r >> 2) * 8 + slot * 4 + (r & 3);
                S[wv * RW + ch * RP + b * 32 + col] = acc[b][r];
            }
        __syncthreads();
        const size_t hw = (size_t)a.ho * a.wo;
        float* yo = a.y + ((size_t)tile.img * a.k + (size_t)tile.kt * 32) * hw + (size_t)tile.m0 * a.wo;
        for (int p = tid; p < tile.npix; p += kBandThreads) {
            float* yp = yo + p + band_image_skip(a, p);
#pragma unroll 4
            for (int ch = 0; ch < 32; ++ch) {
                const int e = ch * RP + p;
                yp[(size_t)ch * hw] = ((S[e] + S[e + RW]) + S[e + 2 * RW]) + S[e + 3 * RW];
            }
        }
    } else {
        // The ks = 1 wave of each channel block leaves its partial sums in
        // LDS (R[block][channel][pixel]); the ks = 0 wave adds them, P0 + P1,
        // and stores the band's valid pixels from its registers.
        float* R = S + cb * RW;
        if (ks > 0) {
#pragma unroll
            for (int b = 0; b < NB; ++b)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int ch = (r >> 2) * 8 + slot * 4 + (r & 3);
                    R[ch * RP + b * 32 + col] = acc[b][r];
                }
        }
        __syncthreads();
        if (ks == 0) {
            const size_t hw = (size_t)a.ho * a.wo;
            float* yo = a.y + ((size_t)tile.img * a.k + (size_t)(tile.kt * CB + cb) * 32) * hw +
                        (size_t)tile.m0 * a.wo;
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                const int p = b * 32 + col;
                float* yp = yo + p + band_image_skip(a, p);
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int ch = (r >> 2) * 8 + slot * 4 + (r & 3);
                    const float v = acc[b][r] + R[ch * RP + p];
                    if (p < tile.npix) yp[(size_t)ch * hw] = v;
                }
            }
        }
    }
}

// The two-way split (KS = 2, 3x3, 64 output channels) with two waves per
// SIMD: waves w and w + 4 take the same 32 output channels and half of the
// chunk's pairs, for the band's first ceil(NB/2) pixel blocks (w < 4) or the
// other NB - ceil(NB/2) (w >= 4), so each SIMD always has a second wave to
// issue while one waits.  Every wave stages one channel slot per chunk.
// Otherwise as conv_f32_band_kernel (same staging modes, same LDS layout,
// same matrix-core sequence per output, P0 + P1 in the same order), so its
// outputs are bitwise those of the one-wave-per-SIMD kernel.
template <int FH, int FW, int NB, int MODE>
__global__ __launch_bounds__(2 * kBandThreads, 1) void conv_f32_band8_kernel(F32BandArgs a) {
    constexpr int T = FH * FW;
    constexpr int PP = 2;                            // channel pairs of a chunk per wave
    constexpr int STEPS = PP * T;                    // k-steps of a chunk per wave
    constexpr int NJ = band_copies(MODE) / 2;        // copies per wave per chunk: one slot
    constexpr int DPT = (NJ + STEPS - 1) / STEPS;    // copies issued after each k-step
    constexpr int PAIR_B = 2 * kBandSlot * 4;        // LDS bytes from one pair's slots to the next
    constexpr int NB0 = (NB + 1) / 2;                // pixel blocks of the waves 0-3
    extern __shared__ __align__(16) float S[];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);   // 0 .. 7
    const int ph = wv >> 2, cb = (wv >> 1) & 1, ks = wv & 1;
    const int bid = a.xcd_remap ? (int)(blockIdx.x & 7) * (a.grid >> 3) + (int)(blockIdx.x >> 3)
                                : (int)blockIdx.x;
    const BandTile tile = band_tile(a, bid);
    const int slot = lane >> 5, col = lane & 31;
    const int kout = (tile.kt * 2 + cb) * 32 + col;
    const __amdgpu_buffer_rsrc_t wres = band_rsrc(a.wt, (uint32_t)((size_t)a.k * a.c * T * 4));
    const int wlane = ((kout * a.c) + 2 * ks * PP + slot) * T * 4;
    const size_t img_elems = (size_t)a.c * a.plane_src;
    const __amdgpu_buffer_rsrc_t sres =
        band_rsrc(a.src + (size_t)tile.img * img_elems, (uint32_t)(tile.nimg * img_elems * 4));
    const int plane_bytes = a.plane_src * 4;
    uint32_t sofs[NJ];
#pragma unroll
    for (int s = 0; s < NJ; ++s) sofs[s] = band_source(a, tile, MODE, FH, s, lane);

    // Copy j of chunk ch into stage ST: channel slot wv, part j.
    auto copy = [&](int j, int ch, auto st_tag) {
        constexpr int ST = decltype(st_tag)::value;
        if (MODE == kBandRaw && j >= a.rgroups) return;
        const uint32_t cbytes = (uint32_t)((ch * kBandChunk + wv) * plane_bytes);
        char* dst = reinterpret_cast<char*>(S) + ST * kBandStageBytes + band_dest_slot(a, MODE, wv, j);
        if (MODE != kBandRaw || lane < a.rrpi * a.rlanes) {
#if defined(__HIP_DEVICE_COMPILE__)   // (16-byte LDS copies exist on gfx950 only; the host pass checks them too)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(sres, (lds_void*)dst,
                                                     MODE == kBandWide || MODE == kBandRaw ? 16 : 4,
                                                     sofs[j] + cbytes, 0, 0, 0);
#endif
        }
    };
    auto load_filter = [&](int ch, int q) {   // k-step q = pp*T + t
        const int pp = q / T, t = q - pp * T;
        return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                             wres, wlane + (2 * pp * T + t) * 4, ch * kBandChunk * T * 4, 0));
    };
    auto land = [&]() {
        __builtin_amdgcn_s_waitcnt(0x0F70);
        __syncthreads();
    };

    // The whole kernel for NBW pixel blocks starting at block B0.
    auto body = [&](auto nbw_tag) {
        constexpr int NBW = decltype(nbw_tag)::value;
        const int B0 = ph * NB0;
        uint32_t bb[NBW];
#pragma unroll
        for (int b = 0; b < NBW; ++b) bb[b] = band_window(a, tile, FH, 2 * ks * PP + slot, lane, B0 + b);
        float fa0[STEPS], fa1[STEPS];
        f32x16 acc[NBW];
#pragma unroll
        for (int b = 0; b < NBW; ++b)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[b][r] = 0.0f;
        auto chunk = [&](auto st_tag, const float (&fa)[STEPS], float (&fn)[STEPS], int ch) {
            constexpr int ST = decltype(st_tag)::value;
            const char* base = reinterpret_cast<const char*>(S) + ST * kBandStageBytes;
            float bv[2][NBW];
            auto read_step = [&](int q, float (&dst)[NBW]) {
                const int pp = q / T, t = q - pp * T;
                const int u = t / FW, v = t - u * FW;
                const int off = pp * PAIR_B + (MODE == kBandRaw ? (u * a.rpitch + v) * 4 : (v * FH + u) * 4);
#pragma unroll
                for (int b = 0; b < NBW; ++b) dst[b] = *reinterpret_cast<const float*>(base + bb[b] + off);
            };
            read_step(0, bv[0]);
#pragma unroll
            for (int q = 0; q < STEPS; ++q) {
                if (q + 1 < STEPS) read_step(q + 1, bv[(q + 1) & 1]);
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int b = 0; b < NBW; ++b)
                    acc[b] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[q], bv[q & 1][b], acc[b], 0, 0, 0);
                BAND_PIN_VMEM();
#pragma unroll
                for (int d = 0; d < DPT; ++d)
                    if (q * DPT + d < NJ) copy(q * DPT + d, ch + 1, std::integral_constant<int, 1 - ST>());
                fn[q] = load_filter(ch + 1, q);
                __builtin_amdgcn_sched_barrier(0);
            }
        };
#pragma unroll
        for (int j = 0; j < NJ; ++j) copy(j, 0, std::integral_constant<int, 0>());
#pragma unroll
        for (int q = 0; q < STEPS; ++q) fa0[q] = load_filter(0, q);
        land();
        for (int ch = 0; ch < a.nchunks; ch += 2) {   // nchunks is even
            chunk(std::integral_constant<int, 0>(), fa0, fa1, ch);
            land();
            chunk(std::integral_constant<int, 1>(), fa1, fa0, ch + 1);
            land();
        }
        // P0 + P1 through LDS, R[block][channel][pixel], as the one-wave kernel
        constexpr int RP = NB * 32;
        constexpr int RW = 32 * RP;
        float* R = S + cb * RW;
        if (ks > 0) {
#pragma unroll
            for (int b = 0; b < NBW; ++b)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int ch = (r >> 2) * 8 + slot * 4 + (r & 3);
                    R[ch * RP + (B0 + b) * 32 + col] = acc[b][r];
                }
        }
        __syncthreads();
        if (ks == 0) {
            const size_t hw = (size_t)a.ho * a.wo;
            float* yo = a.y + ((size_t)tile.img * a.k + (size_t)(tile.kt * 2 + cb) * 32) * hw + (size_t)tile.m0 * a.wo;
#pragma unroll
            for (int b = 0; b < NBW; ++b) {
                const int p = (B0 + b) * 32 + col;
                float* yp = yo + p + band_image_skip(a, p);
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int ch = (r >> 2) * 8 + slot * 4 + (r & 3);
                    const float v = acc[b][r] + R[ch * RP + p];
                    if (p < tile.npix) yp[(size_t)ch * hw] = v;
                }
            }
        }
    };
    if (ph == 0)
        body(std::integral_constant<int, NB0>());
    else
        body(std::integral_constant<int, NB - NB0>());
}

// Layers with few input channels (C = 3: the 7x7 stride-2 stems, the 11x11
// stride-4 and 3x3 first layers): the whole reduction of a band is C*Fh*Fw
// elements, so a band's C strips are staged at once.  The kernel is
// persistent: one workgroup per CU walks through a run of consecutive bands
// (same output channels and image, neighbouring rows), with the strips of
// band b + 1 copied into a second LDS buffer while band b is multiplied, and
// band b - 1's outputs stored from registers between band b's MFMAs, so that
// no phase of a band waits for memory.  Fused, the band's zero-padded input
// rows take the strips' place: window element (u, v) of output pixel (m, n)
// is input row m*sh + u, column n*sw + v - pw, a fixed offset from the
// window's start, as in the window tensor.  The filter values stay in
// registers across the run; they are reloaded only where the run crosses
// into the next group of output channels.  The MFMA's two k-slots take
// filter rows u and u + Fh - ceil(Fh/2) of one channel and tap column (one
// LDS read: the second slot is the first plus Fh - ceil(Fh/2) rows),
// u < ceil(Fh/2); for odd Fh the middle row comes up in both slots and the
// second slot's copy gets zero weights, so every read stays inside the
// pixel's window.  Waves (cb, ks): 2 blocks of 32 output channels x 2
// halves of the C*ceil(Fh/2)*Fw k-steps; with WPS = 2 waves w and w + 4 take
// wave w's share for the first ceil(NB/2) pixel blocks and the rest, two
// waves per SIMD, and the staging copies go round the 8 waves.
template <int C, int FH, int FW, int NB, int MODE, int WPS>
__global__ __launch_bounds__(WPS * kBandThreads, 1) void conv_f32_band_small_c_kernel(F32BandArgs a) {
    constexpr int HU = (FH + 1) / 2;
    constexpr int S = smallc_steps(C, FH, FW);   // k-steps of the whole reduction
    constexpr int SW = (S + 1) / 2;     // k-steps of the first half (the second takes S - SW)
    constexpr int RP = NB * 32;
    constexpr int RW = 32 * RP;         // floats of one block's partial sums
    constexpr bool GATHER = MODE == kBandGather;
    constexpr int NT = WPS * kBandThreads, NWV = 4 * WPS;   // threads, waves
    constexpr int NB0 = (NB + WPS - 1) / WPS;   // pixel blocks of the waves 0-3 (the rest: waves 4-7)
    extern __shared__ __align__(16) float L[];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int ph = wv >> 2, cb = (wv >> 1) & 1, ks = wv & 1;
    const int slot = lane >> 5, col = lane & 31;
    // LDS: two strip buffers (unfused) or two buffers of zero-padded raw
    // input rows (fused), then the partial sums of the two blocks
    const int buf_f = GATHER ? C * a.rrows * a.rpitch : C * a.slotf;   // floats per buffer
    float* R = L + 2 * buf_f + cb * RW;
    const int b0 = (int)blockIdx.x * a.per_wg;
    const int b1 = b0 + a.per_wg < a.total ? b0 + a.per_wg : a.total;
    const __amdgpu_buffer_rsrc_t wres = band_rsrc(a.wt, (uint32_t)((size_t)a.k * C * FH * FW * 4));
    const size_t img_elems = (size_t)C * a.plane_src;

    // Unfused: the C strips of band bid (runs of the window tensor) into
    // strip buffer buf, parts of 256 (wide) or 64 elements; copy c*np + sp
    // goes to wave (c*np + sp) mod 4.  Copies past the strip read zeros.
    auto issue_strips = [&](int bid, int buf) {
        const BandTile t = smallc_tile(a, bid);
        const __amdgpu_buffer_rsrc_t sres = band_rsrc(a.src + (size_t)t.img * img_elems, (uint32_t)(img_elems * 4));
        const int np = smallc_parts(a, t);
#pragma unroll
        for (int c = 0; c < C; ++c) {
            for (int sp = (wv - c * np) & (NWV - 1); sp < np; sp += NWV) {
                const uint32_t off = band_source(a, t, MODE, FH, sp, lane);
                char* dst =
                    reinterpret_cast<char*>(L) + (buf * buf_f + c * a.slotf + sp * (MODE == kBandWide ? 256 : 64)) * 4;
                const uint32_t voff = off == kBandOutside ? off : off + (uint32_t)(c * a.plane_src * 4);
#if defined(__HIP_DEVICE_COMPILE__)   // (16-byte LDS copies exist on gfx950 only; the host pass checks them too)
                if constexpr (MODE == kBandWide)
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(sres, (lds_void*)dst, 16, voff, 0, 0, 0);
                else
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(sres, (lds_void*)dst, 4, voff, 0, 0, 0);
#endif
            }
        }
    };
    // Fused: the rrows input rows of band bid (rows m0*sh - ph .., zero
    // outside the image) of the C channels into raw buffer buf, columns
    // 0..W-1 at rlpad, in rparts copies per row (16-byte pieces, or 4-byte
    // ones when rows are not whole vectors); row c*rrows + r goes to wave
    // (c*rrows + r) mod 4.  The pad columns around them were zeroed once and
    // are never written.  With them the raw rows hold every window element
    // of the band at a fixed offset from the window's start, so the k-steps
    // read them as they read the window tensor's strips.
    auto issue_raw = [&](int bid, int buf) {
        const BandTile t = smallc_tile(a, bid);
        const __amdgpu_buffer_rsrc_t sres = band_rsrc(a.src + (size_t)t.img * img_elems, (uint32_t)(img_elems * 4));
        const int y0 = t.m0 * a.sh - a.ph;
        const int per = a.rawwide ? 4 : 1;
#pragma unroll
        for (int c = 0; c < C; ++c) {
            for (int r = (wv - c * a.rrows) & (NWV - 1); r < a.rrows; r += NWV) {
                const int yy = y0 + r;   // wave-uniform
                const uint32_t rowoff = (uint32_t)((c * a.h + yy) * a.w) * 4u;
                const bool in = yy >= 0 && yy < a.h;
                const int dst0 = (buf * buf_f + (c * a.rrows + r) * a.rpitch + a.rlpad) * 4;
                for (int pr = 0; pr < a.rparts; ++pr) {
                    const int xx = pr * 64 * per + lane * per;   // first column of this lane
                    if (xx < a.w) {
                        const uint32_t voff = in ? rowoff + (uint32_t)xx * 4u : kBandOutside;
                        char* dst = reinterpret_cast<char*>(L) + dst0 + pr * 256 * per;
#if defined(__HIP_DEVICE_COMPILE__)
                        if (a.rawwide)
                            __builtin_amdgcn_raw_ptr_buffer_load_lds(sres, (lds_void*)dst, 16, voff, 0, 0, 0);
                        else
                            __builtin_amdgcn_raw_ptr_buffer_load_lds(sres, (lds_void*)dst, 4, voff, 0, 0, 0);
#endif
                    }
                }
            }
        }
    };
    if constexpr (GATHER) {
        // the pad columns (rlpad before each raw row, rpitch - rlpad - W after)
        // of every raw row of both buffers
        const int padc = a.rpitch - a.w;
        for (int i = tid; i < 2 * C * a.rrows * padc; i += NT) {
            const int row = i / padc, k = i - row * padc;
            L[row * a.rpitch + (k < a.rlpad ? k : a.w + k)] = 0.0f;
        }
    }
    // Filter values of this wave's k-steps q = ks*SW + i for the output
    // channels of group kt: the (channel, row, column) of each k-slot's
    // element (smallc_step; zero for the repeated middle row, past the last
    // step, and for output channels past K, whose offsets lie past the
    // filter).  q is compile-time per half, so each load is a per-lane base
    // plus an immediate, the k-slot a select.
    auto load_filter_half = [&](auto ks_tag, int kt, float (&f)[SW]) {
        constexpr int KSI = decltype(ks_tag)::value;
        const int kout = (kt * 2 + cb) * 32 + col;
        // slot 1's element lies one channel (pair steps) or Fh - HU rows (the
        // last channel's steps) after slot 0's
        const uint32_t base = (uint32_t)(kout * C * FH * FW * 4);
        const uint32_t bpair = base + (uint32_t)(slot * FH * FW * 4), blast = base + (uint32_t)(slot * (FH - HU) * FW * 4);
#pragma unroll
        for (int i = 0; i < SW; ++i) {
            const int q = KSI * SW + i;
            if (q >= S) {
                f[i] = 0.0f;
                continue;
            }
            const SmallCStep s0 = smallc_step(C, FH, FW, q, 0), s1 = smallc_step(C, FH, FW, q, 1);
            const uint32_t imm = (uint32_t)(((s0.c * FH + s0.u) * FW + s0.v) * 4);
            uint32_t off = (s0.pair ? bpair : blast) + imm;
            if (s1.zero) off = slot ? kBandOutside : off;   // slot 1 would repeat a slot-0 row
            f[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(wres, off, 0, 0));
        }
    };
    auto load_filter = [&](int kt, float (&f)[SW]) {
        if (ks == 0)
            load_filter_half(std::integral_constant<int, 0>(), kt, f);
        else
            load_filter_half(std::integral_constant<int, 1>(), kt, f);
    };

    // The rest for NBW pixel blocks from block B0 (this wave's share).
    auto body = [&](auto nbw_tag) {
    constexpr int NBW = decltype(nbw_tag)::value;
    constexpr int NOUT = NBW * 16;       // output registers per lane
    constexpr int SPS = (2 * NOUT + SW - 1) / SW;   // stores issued per k-step (done halfway through)
    const int B0 = ph * NB0;
    // y through a buffer resource over the previous band's image: a store
    // whose offset lies past its end (pixels past the band, or no previous
    // band yet) is dropped
    const size_t hw = (size_t)a.ho * a.wo;
    __amdgpu_buffer_rsrc_t yres = band_rsrc(a.y, 0u);
    float fa[SW];
    f32x16 acc[NBW], out[NBW];
    // byte offset in y of the previous band's channel 0, pixel (lane, block);
    // the channel adds ch*hw*4 (scalar)
    uint32_t ybase[NBW];
#pragma unroll
    for (int b = 0; b < NBW; ++b) {
        ybase[b] = kBandOutside;
#pragma unroll
        for (int r = 0; r < 16; ++r) out[b][r] = 0.0f;
    }

    int kt_loaded = smallc_tile(a, b0).kt;
    load_filter(kt_loaded, fa);
    __builtin_amdgcn_s_waitcnt(0x0F70);
    if constexpr (GATHER)
        issue_raw(b0, 0);
    else
        issue_strips(b0, 0);
    for (int bid = b0; bid < b1; ++bid) {
        const int cur = (bid - b0) & 1;
        // band bid's strips (raw rows) have landed, and the stores issued
        // during band bid - 1; every wave is done with the buffers band
        // bid - 1 read and with R
        __builtin_amdgcn_s_waitcnt(0x0F70);
        __syncthreads();
        const BandTile tile = smallc_tile(a, bid);
        if (tile.kt != kt_loaded) {   // wave-uniform; waited for here, before the next copies are issued
            kt_loaded = tile.kt;
            load_filter(kt_loaded, fa);
            __builtin_amdgcn_s_waitcnt(0x0F70);
        }
        if (bid + 1 < b1) {
            if constexpr (GATHER)
                issue_raw(bid + 1, cur ^ 1);
            else
                issue_strips(bid + 1, cur ^ 1);
        }
        // byte offset of each block's window for this lane's k-slot: in the
        // channel-pair steps (slot 1 one channel further), and in the last
        // channel's steps (slot 1 Fh - HU rows further); the step's channel
        // and tap add a uniform offset
        uint32_t bp[NBW], bl[NBW];
#pragma unroll
        for (int b = 0; b < NBW; ++b) {
            if constexpr (GATHER) {
                const uint32_t r0 = smallc_raw_window(a, tile, FH, lane, B0 + b) + (uint32_t)(cur * buf_f) * 4u;
                bp[b] = r0 + (uint32_t)(slot * a.rrows * a.rpitch) * 4u;
                bl[b] = r0 + (uint32_t)(slot * (FH - HU) * a.rpitch) * 4u;
            } else {
                const uint32_t w0 = smallc_window(a, tile, FH, lane, B0 + b) + (uint32_t)(cur * buf_f) * 4u;
                bp[b] = w0 + (uint32_t)(slot * a.slotf) * 4u;
                bl[b] = w0 + (uint32_t)((C - 1) * a.slotf + slot * (FH - HU)) * 4u;
            }
        }
#pragma unroll
        for (int b = 0; b < NBW; ++b)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[b][r] = 0.0f;

        // The k-steps of half KSI (the immediates of the LDS reads follow the
        // step, so each half is its own code); the ks = 0 waves store the
        // previous band's sums, SPS values per step.
        auto run = [&](auto ks_tag) {
            constexpr int KSI = decltype(ks_tag)::value;
            constexpr int Q0 = KSI * SW, NQ = KSI == 0 ? SW : S - SW;
            float bv[2][NBW];
            auto read_step = [&](int i, float (&dst)[NBW]) {
                const SmallCStep s0 = smallc_step(C, FH, FW, Q0 + i, 0);   // slot 0's element
                const char* Lb = reinterpret_cast<const char*>(L);
                // uniform offset of slot 0's element from the slot's base
                int off;
                if constexpr (GATHER)
                    off = ((s0.pair ? s0.c * a.rrows : 0) + s0.u) * a.rpitch * 4 + s0.v * 4;
                else
                    off = ((s0.pair ? s0.c * a.slotf : 0) + s0.v * FH + s0.u) * 4;
                if (!s0.pair && GATHER) off += (C - 1) * a.rrows * a.rpitch * 4;
#pragma unroll
                for (int b = 0; b < NBW; ++b)
                    dst[b] = *reinterpret_cast<const float*>(Lb + (s0.pair ? bp[b] : bl[b]) + off);
            };
            read_step(0, bv[0]);
#pragma unroll
            for (int i = 0; i < NQ; ++i) {
                if (i + 1 < NQ) read_step(i + 1, bv[(i + 1) & 1]);
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int b = 0; b < NBW; ++b)
                    acc[b] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[i], bv[i & 1][b], acc[b], 0, 0, 0);
                if constexpr (KSI == 0) {
#pragma unroll
                    for (int e = i * SPS; e < (i + 1) * SPS && e < NOUT; ++e) {
                        const int b = e / 16, r = e % 16;
                        const int chs = (r >> 2) * 8 + (r & 3);   // + slot*4, in ybase
                        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(elem(out[b], r)), yres, ybase[b],
                                                              (int)(chs * hw * 4), 0);
                    }
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        };
        if (ks == 0)
            run(std::integral_constant<int, 0>());
        else
            run(std::integral_constant<int, 1>());

        // The ks = 1 wave of each block leaves its partial sums in R; the
        // ks = 0 wave adds them, P0 + P1, into `out`.  The barrier waits for
        // the LDS writes only (counter lgkmcnt 0): the next band's copies and
        // this band's stores stay in flight.
        if (ks > 0) {
#pragma unroll
            for (int b = 0; b < NBW; ++b)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int ch = (r >> 2) * 8 + slot * 4 + (r & 3);
                    R[ch * RP + (B0 + b) * 32 + col] = acc[b][r];
                }
        }
        __builtin_amdgcn_s_waitcnt(0xC07F);
        asm volatile("s_barrier" ::: "memory");
        if (ks == 0) {
#pragma unroll
            for (int b = 0; b < NBW; ++b)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int ch = (r >> 2) * 8 + slot * 4 + (r & 3);
                    out[b][r] = acc[b][r] + R[ch * RP + (B0 + b) * 32 + col];
                }
            yres = band_rsrc(a.y + (size_t)tile.img * a.k * hw, (uint32_t)((size_t)a.k * hw * 4));
            const uint32_t y0 = (uint32_t)((((size_t)(tile.kt * 2 + cb) * 32 + slot * 4) * hw + (size_t)tile.m0 * a.wo) * 4);
            // (a block of output channels past K, K = 32 mod 64, has zero
            // weights and stores nothing)
            const bool kin = (tile.kt * 2 + cb) * 32 < a.k;
#pragma unroll
            for (int b = 0; b < NBW; ++b) {
                const int p = (B0 + b) * 32 + col;
                ybase[b] = kin && p < tile.npix ? y0 + (uint32_t)p * 4u : kBandOutside;
            }
        }
    }
    // the last band's sums
    if (ks == 0) {
#pragma unroll
        for (int e = 0; e < NOUT; ++e) {
            const int b = e / 16, r = e % 16;
            const int chs = (r >> 2) * 8 + (r & 3);
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(elem(out[b], r)), yres, ybase[b],
                                                  (int)(chs * hw * 4), 0);
        }
    }
    };
    if constexpr (WPS == 1) {
        body(std::integral_constant<int, NB>());
    } else {
        if (ph == 0)
            body(std::integral_constant<int, NB0>());
        else
            body(std::integral_constant<int, NB - NB0>());
    }
}

template <int FH, int FW, int NB, int MODE, int KS>
void launch_band_v(const F32BandArgs& a, int64_t lds, hipStream_t stream) {
    if (lds > 64 * 1024)
        (void)hipFuncSetAttribute((const void*)conv_f32_band_kernel<FH, FW, NB, MODE, KS>,
                                  hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL((conv_f32_band_kernel<FH, FW, NB, MODE, KS>), dim3((unsigned)a.grid), dim3(kBandThreads),
                       (size_t)lds, stream, a);
}

template <int FH, int FW, int NB, int MODE>
void launch_band8_v(const F32BandArgs& a, int64_t lds, hipStream_t stream) {
    if (lds > 64 * 1024)
        (void)hipFuncSetAttribute((const void*)conv_f32_band8_kernel<FH, FW, NB, MODE>,
                                  hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL((conv_f32_band8_kernel<FH, FW, NB, MODE>), dim3((unsigned)a.grid), dim3(2 * kBandThreads),
                       (size_t)lds, stream, a);
}

template <int FH, int FW, int NB>
void launch_band8_nb(const F32BandArgs& a, int64_t lds, hipStream_t stream) {
    if (a.mode == kBandRaw)
        launch_band8_v<FH, FW, NB, kBandRaw>(a, lds, stream);
    else if (a.mode == kBandGather)
        launch_band8_v<FH, FW, NB, kBandGather>(a, lds, stream);
    else if (a.mode == kBandNarrow)
        launch_band8_v<FH, FW, NB, kBandNarrow>(a, lds, stream);
    else
        launch_band8_v<FH, FW, NB, kBandWide>(a, lds, stream);
}

template <int FH, int FW, int NB, int KS>
void launch_band_nb(const F32BandArgs& a, int64_t lds, hipStream_t stream) {
    if (a.mode == kBandRaw)
        launch_band_v<FH, FW, NB, kBandRaw, KS>(a, lds, stream);
    else if (a.mode == kBandGather)
        launch_band_v<FH, FW, NB, kBandGather, KS>(a, lds, stream);
    else if (a.mode == kBandNarrow)
        launch_band_v<FH, FW, NB, kBandNarrow, KS>(a, lds, stream);
    else
        launch_band_v<FH, FW, NB, kBandWide, KS>(a, lds, stream);
}

// Pixel blocks per band that the kernels are built for.
constexpr int kBandNb4Min = 4, kBandNb4Max = 7;     // four-way split
constexpr int kBandNb2Min = 11, kBandNb2Max = 14;   // two-way split (3x3), and:
constexpr int kBandNb2Pair = 9;                      // two whole images of 144 pixels

constexpr int kBandMaxRounds = 4;   // rounds of 256 workgroups, unless a workgroup's work is long:
constexpr double kBandLongMacs = 12e6;   // multiply-adds per workgroup

bool band_shape_ok(const Geometry& g, int ks, int nb) {
    if (!band_nb_compiled(ks, nb)) return false;
    if (ks == 4) return (g.fh == 3 && (g.fw == 3 || g.fw == 5)) || (g.fh == 5 && g.fw == 5);
    return g.fh == 3 && g.fw == 3 && g.k % 64 == 0;
}

}  // namespace

bool band_nb_compiled(int ks, int nb) {
    if (ks == 4) return nb >= kBandNb4Min && nb <= kBandNb4Max;
    return ks == 2 && (nb == kBandNb2Pair || (nb >= kBandNb2Min && nb <= kBandNb2Max));
}

F32BandPlan plan_band_f32(const Geometry& g) {
    F32BandPlan best;
    if (g.elem != 4 || g.c % (2 * kBandChunk) || g.k % 32) return best;
    if (g.c * g.h * g.w * 4 >= (int64_t(1) << 30) || g.c * g.ho * g.row_len * 4 >= (int64_t(1) << 30) ||
        g.k * g.c * g.taps * 4 >= (int64_t(1) << 31) || g.n * g.k * g.ho * g.wo >= (int64_t(1) << 31))
        return best;
    // useful matrix-core work (32x32 blocks of output x chunk pairs) over the
    // work the launch occupies: whole rounds of 256 workgroups, each with 4
    // waves of NB blocks x PP pairs
    const double useful = (double)g.n * (g.k / 32) * (double)(g.ho * g.wo) / 32.0 * 4.0;
    for (int ks : {4, 2}) {
        const int pp = 4 / ks;
        for (int64_t rows = g.ho; rows >= 1; --rows) {
            if (rows * g.row_len + 3 > 64 * kBandMaxSeg) continue;
            const int64_t nb = (rows * g.wo + 31) / 32;
            if (!band_shape_ok(g, ks, (int)nb)) continue;
            const int64_t nbands = (g.ho + rows - 1) / rows;
            const int64_t grid = g.n * nbands * (g.k / (32 * (4 / ks)));
            if (grid > 0x7fffffff) continue;
            const int64_t rounds = (grid + 255) / 256;
            // many short rounds: the tile kernels, which overlap one
            // workgroup's staging with another's multiplies, do better
            // (with long ones, staging a band is a small share of its work)
            const double wg_macs = (double)(4 / ks) * 32 * nb * 32 * g.c * g.taps;
            if (rounds > kBandMaxRounds && wg_macs < kBandLongMacs) continue;
            const double eff = useful / ((double)rounds * 1024.0 * nb * pp);
            if (eff > best.eff + 1e-9) {
                best.ks = ks;
                best.rows = (int)rows;
                best.nb = (int)nb;
                best.ipb = 1;
                best.grid = grid;
                best.eff = eff;
            }
        }
        // bands of several whole images, for feature maps smaller than a
        // band (their strips back to back in a slot, within 2^30 bytes of
        // source per band)
        for (int64_t ipb = 2; ipb <= g.n; ++ipb) {
            if (ipb * g.ho * g.row_len + 3 > 64 * kBandMaxSeg) break;
            const int64_t nb = (ipb * g.ho * g.wo + 31) / 32;
            if (ipb * g.c * std::max(g.h * g.w, g.ho * g.row_len) * 4 >= (int64_t(1) << 30)) break;
            if (!band_shape_ok(g, ks, (int)nb)) continue;
            const int64_t grid = (g.n + ipb - 1) / ipb * (g.k / (32 * (4 / ks)));
            const int64_t rounds = (grid + 255) / 256;
            const double wg_macs = (double)(4 / ks) * 32 * nb * 32 * g.c * g.taps;
            if (rounds > kBandMaxRounds && wg_macs < kBandLongMacs) continue;
            const double eff = useful / ((double)rounds * 1024.0 * nb * pp);
            if (eff > best.eff + 1e-9) {
                best.ks = ks;
                best.rows = (int)g.ho;
                best.nb = (int)nb;
                best.ipb = (int)ipb;
                best.grid = grid;
                best.eff = eff;
            }
        }
    }
    if (best.eff < 0.85) return F32BandPlan();
    // partial sums: four per block of 32 channels (four-way split), or one
    // per block of the two
    const int64_t red = (int64_t)(best.ks == 4 ? 4 : 2) * 32 * best.nb * 32 * 4;
    best.lds_bytes = std::max<int64_t>(2 * kBandStageBytes, red);
    if (best.lds_bytes > kConvLdsMaxBytes) return F32BandPlan();
    best.ok = true;
    return best;
}

F32BandArgs band_args_f32(const Geometry& g, const F32BandPlan& p, bool fused, const void* src, const void* w,
                          float* y) {
    F32BandArgs a;
    a.src = static_cast<const float*>(src);
    a.wt = static_cast<const float*>(w);
    a.y = y;
    a.n = (int)g.n; a.c = (int)g.c; a.h = (int)g.h; a.w = (int)g.w; a.k = (int)g.k;
    a.sh = (int)g.sh; a.sw = (int)g.sw; a.ph = (int)g.ph; a.pw = (int)g.pw;
    a.ho = (int)g.ho; a.wo = (int)g.wo;
    a.row_len = (int)g.row_len;
    a.div_row = make_fastdiv((uint32_t)g.row_len);
    a.div_wo = make_fastdiv((uint32_t)g.wo);
    a.div_ho = make_fastdiv((uint32_t)g.ho);
    a.plane_src = fused ? (int)(g.h * g.w) : (int)(g.ho * g.row_len);
    a.rows = p.rows;
    a.ipb = p.ipb;
    a.nbands = p.ipb > 1 ? 1 : (int)((g.ho + p.rows - 1) / p.rows);
    a.ks = p.ks;
    a.nkt = (int)(g.k / (32 * (4 / p.ks)));
    a.nchunks = (int)(g.c / kBandChunk);
    a.grid = (int)p.grid;
    a.xcd_remap = (p.grid % 8 == 0 && p.grid > 8) ? 1 : 0;
    // 16-byte copies need 16-byte aligned planes
    const bool aligned = ((uintptr_t)src & 15) == 0 && (g.ho * g.row_len) % 4 == 0;
    a.rrows = a.rpitch = a.rlpad = a.rlanes = a.rrpi = a.rgroups = 0;
    a.rawwide = a.rparts = 0;
    a.mode = fused ? (p.ipb == 1 && band_raw_mode(g, p.rows, src, &a) ? kBandRaw : kBandGather)
                   : aligned ? kBandWide : kBandNarrow;
    a.slotf = 0;
    a.total = a.grid;
    a.per_wg = 1;
    return a;
}

bool band_raw_mode(const Geometry& g, int rows, const void* x, F32BandArgs* a) {
    if (g.w % 4 || ((uintptr_t)x & 15)) return false;
    const int64_t rlpad = (g.pw + 3) / 4 * 4;
    const int64_t reach = std::max(g.w, (g.wo - 1) * g.sw + g.fw - g.pw);   // columns 0 .. reach-1
    int64_t rlanes = (rlpad + reach + 3) / 4;
    // consecutive output rows of a block (sh raw rows apart) in other banks
    if ((rlanes * 4 * g.sh) % 64 == 0) ++rlanes;
    if (rlanes > 64) return false;
    const int64_t rrpi = 64 / rlanes, rrows = (rows - 1) * g.sh + g.fh;
    const int64_t rgroups = (rrows + rrpi - 1) / rrpi;
    if (rgroups > kBandRawGroups || rgroups * rrpi * rlanes * 4 > kBandSlot) return false;
    a->rrows = (int)rrows;
    a->rpitch = (int)(rlanes * 4);
    a->rlpad = (int)rlpad;
    a->rlanes = (int)rlanes;
    a->rrpi = (int)rrpi;
    a->rgroups = (int)rgroups;
    return true;
}

int launch_conv_f32_band(const Geometry& g, const F32BandPlan& p, bool fused, const void* src, const void* w,
                         float* y, hipStream_t stream) {
    const F32BandArgs a = band_args_f32(g, p, fused, src, w, y);
    const int64_t lds = p.lds_bytes;
    if (p.ks == 2) {
        // two waves per SIMD (with the four-way split they were slower:
        // 3-4 pixel blocks per wave)
        if (p.nb == kBandNb2Pair) launch_band8_nb<3, 3, kBandNb2Pair>(a, lds, stream);
        else if (p.nb == 11) launch_band8_nb<3, 3, 11>(a, lds, stream);
        else if (p.nb == 12) launch_band8_nb<3, 3, 12>(a, lds, stream);
        else if (p.nb == 13) launch_band8_nb<3, 3, 13>(a, lds, stream);
        else launch_band8_nb<3, 3, 14>(a, lds, stream);
        return 0;
    }
#define BAND_NB4(FH_, FW_)                                                \
    switch (p.nb) {                                                       \
        case 4: launch_band_nb<FH_, FW_, 4, 4>(a, lds, stream); break;    \
        case 5: launch_band_nb<FH_, FW_, 5, 4>(a, lds, stream); break;    \
        case 6: launch_band_nb<FH_, FW_, 6, 4>(a, lds, stream); break;    \
        default: launch_band_nb<FH_, FW_, 7, 4>(a, lds, stream); break;   \
    }
    if (g.fh == 5) {
        BAND_NB4(5, 5)
    } else if (g.fw == 3) {
        BAND_NB4(3, 3)
    } else {
        BAND_NB4(3, 5)
    }
#undef BAND_NB4
    return 0;
}

namespace {

template <int FH, int NB, int MODE>
void launch_small_c_v(const F32BandArgs& a, int64_t lds, hipStream_t stream) {
    constexpr int C = kSmallCChannels, WPS = kSmallCWavesPerSimd;
    if (lds > 64 * 1024)
        (void)hipFuncSetAttribute((const void*)conv_f32_band_small_c_kernel<C, FH, FH, NB, MODE, WPS>,
                                  hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL((conv_f32_band_small_c_kernel<C, FH, FH, NB, MODE, WPS>), dim3((unsigned)a.grid),
                       dim3(WPS * kBandThreads), (size_t)lds, stream, a);
}

template <int FH, int NB>
void launch_small_c_nb(const F32BandArgs& a, int64_t lds, hipStream_t stream) {
    if (a.mode == kBandGather)
        launch_small_c_v<FH, NB, kBandGather>(a, lds, stream);
    else if (a.mode == kBandNarrow)
        launch_small_c_v<FH, NB, kBandNarrow>(a, lds, stream);
    else
        launch_small_c_v<FH, NB, kBandWide>(a, lds, stream);
}

template <int FH>
void launch_small_c_fh(const F32BandArgs& a, int nb, int64_t lds, hipStream_t stream) {
    switch (nb) {
        case 4: launch_small_c_nb<FH, 4>(a, lds, stream); break;
        case 5: launch_small_c_nb<FH, 5>(a, lds, stream); break;
        case 6: launch_small_c_nb<FH, 6>(a, lds, stream); break;
        default: launch_small_c_nb<FH, 7>(a, lds, stream); break;
    }
}

// LDS floats per channel slot of a band of `rows` rows: the strip, its
// alignment shift and the rounding of the copies to whole 256-element parts.
int64_t small_c_slot(const Geometry& g, int64_t rows) { return (rows * g.row_len + 3 + 255) / 256 * 256; }

// Raw input rows of a band (fused): (rows - 1)*sh + Fh rows per channel,
// each with zero columns before (rlpad >= pw, whole 16-byte vectors so the
// data starts aligned) and after (to the last column a window reaches), the
// pitch whole vectors.
int64_t small_c_rrows(const Geometry& g, int64_t rows) { return (rows - 1) * g.sh + g.fh; }
int64_t small_c_rlpad(const Geometry& g) { return (g.pw + 3) / 4 * 4; }
int64_t small_c_rpitch(const Geometry& g) {
    const int64_t reach = std::max(g.w, (g.wo - 1) * g.sw + g.fw - g.pw);   // columns 0 .. reach-1
    return (small_c_rlpad(g) + reach + 3) / 4 * 4;
}
int64_t small_c_raw(const Geometry& g, int64_t rows) {
    return kSmallCChannels * small_c_rrows(g, rows) * small_c_rpitch(g);
}

}  // namespace

F32BandPlan plan_band_small_c_f32(const Geometry& g) {
    F32BandPlan best;
    if (g.elem != 4 || g.c != kSmallCChannels || g.fh != g.fw || g.k % 32) return best;
    if (g.fh != 3 && g.fh != 7 && g.fh != 11) return best;   // the compiled filter sizes
    // 32-bit buffer offsets; y (stored through a buffer resource) below the
    // dropped-store offset
    if (g.c * g.h * g.w * 4 >= (int64_t(1) << 30) || g.c * g.ho * g.row_len * 4 >= (int64_t(1) << 30) ||
        g.k * g.c * g.taps * 4 >= (int64_t(1) << 31) || g.k * g.ho * g.wo * 4 >= (int64_t(1) << 30))
        return best;
    const int HU = (int)(g.fh + 1) / 2, S = kSmallCChannels * HU * (int)g.fw, SW = (S + 1) / 2;
    // useful MFMA k-steps (pairs of reduction elements) over those the launch
    // occupies: whole workgroups per CU, each 4 waves of NB blocks x SW steps
    const double useful = (double)g.n * (g.k / 32) * (double)(g.ho * g.wo) / 32.0 * (g.c * g.taps / 2.0);
    for (int64_t rows = 1; rows <= g.ho; ++rows) {
        const int64_t nb = (rows * g.wo + 31) / 32;
        if (nb < 4 || nb > 7) continue;
        // two strip buffers (unfused) or two buffers of raw input rows
        // (fused), followed by the partial sums of the two channel blocks
        const int64_t slot = small_c_slot(g, rows), red = 2 * 32 * nb * 32 * 4;
        const int64_t lds = std::max(2 * kSmallCChannels * slot, 2 * small_c_raw(g, rows)) * 4 + red;
        if (lds > kConvLdsMaxBytes) continue;
        const int64_t nbands = (g.ho + rows - 1) / rows;
        const int64_t total = g.n * nbands * ((g.k + 63) / 64);
        if (total > 0x7fffffff) continue;
        const int64_t per_wg = (total + 255) / 256;
        const double eff = useful / ((double)per_wg * 256.0 * 4.0 * nb * SW);
        if (eff > best.eff + 1e-9) {
            best.ks = 2;
            best.rows = (int)rows;
            best.nb = (int)nb;
            best.grid = (total + per_wg - 1) / per_wg;
            best.eff = eff;
            best.lds_bytes = lds;
        }
    }
    if (best.eff < 0.55) return F32BandPlan();
    best.ok = true;
    return best;
}

F32BandArgs band_args_small_c_f32(const Geometry& g, const F32BandPlan& p, bool fused, const void* src,
                                  const void* w, float* y) {
    F32BandArgs a = band_args_f32(g, p, fused, src, w, y);
    if (fused) a.mode = kBandGather;   // (this kernel's fused staging is its own raw-row copy)
    a.rlanes = a.rrpi = a.rgroups = 0;
    a.nkt = (int)((g.k + 63) / 64);   // K = 32 mod 64: the last group's second block idles
    a.nchunks = 1;
    a.slotf = (int)small_c_slot(g, p.rows);
    a.total = (int)(g.n * a.nbands * a.nkt);
    a.per_wg = (a.total + 255) / 256;
    a.grid = (int)p.grid;
    a.xcd_remap = 0;   // each workgroup walks its own run of bands
    a.rrows = (int)small_c_rrows(g, p.rows);
    a.rpitch = (int)small_c_rpitch(g);
    a.rlpad = (int)small_c_rlpad(g);
    // raw rows by 16-byte copies when every row of x starts on a 16-byte boundary
    a.rawwide = (g.w % 4 == 0 && ((uintptr_t)src & 15) == 0) ? 1 : 0;
    a.rparts = a.rawwide ? (a.w + 255) / 256 : (a.w + 63) / 64;
    return a;
}

int launch_conv_f32_band_small_c(const Geometry& g, const F32BandPlan& p, bool fused, const void* src,
                                 const void* w, float* y, hipStream_t stream) {
    const F32BandArgs a = band_args_small_c_f32(g, p, fused, src, w, y);
    if (g.fh == 3)
        launch_small_c_fh<3>(a, p.nb, p.lds_bytes, stream);
    else if (g.fh == 7)
        launch_small_c_fh<7>(a, p.nb, p.lds_bytes, stream);
    else
        launch_small_c_fh<11>(a, p.nb, p.lds_bytes, stream);
    return 0;
}

}  // namespace im2win
