// fp32 im2win convolution by bands of output rows: a workgroup computes a
// band of rows of one image for 32 or 64 output channels, with all 4 waves
// busy on the same amount of matrix-core work, so that a layer of a few
// hundred workgroups fills the chip without the quantization of fixed
// pixel tiles.
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
//     16-byte aligned.  Fused, every strip element is gathered from x by
//     4-byte LDS DMA with per-lane source offsets computed once per kernel;
//     padding positions carry an offset past the end of the buffer, which
//     the hardware reads as zero;
//   - the filter does not go through LDS: each lane loads its own filter
//     rows (one output channel, one input channel per pair, Fh*Fw taps) of
//     the next chunk into registers while the current chunk is multiplied;
//   - the copies of the next chunk are spread over the taps of the current
//     one, and the windows of the next tap are read before the MFMAs of the
//     current tap, so both latencies hide behind matrix-core work.
// Both variants stage the same values into the same strip positions and run
// the same matrix-core sequence, so their outputs are bitwise identical.
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
        band_rsrc(a.src + (size_t)tile.img * img_elems, (uint32_t)(img_elems * 4));
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
    auto copy = [&](int j, int ch, auto st_tag) {
        constexpr int ST = decltype(st_tag)::value;
        const uint32_t cbytes = (uint32_t)((ch * kBandChunk + 2 * wv + (j & 1)) * plane_bytes);
        char* dst = reinterpret_cast<char*>(S) + ST * kBandStageBytes + band_dest(MODE, wv, j);
#if defined(__HIP_DEVICE_COMPILE__)   // (16-byte LDS copies exist on gfx950 only; the host pass checks them too)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(sres, (lds_void*)dst, MODE == kBandWide ? 16 : 4,
                                                 sofs[j >> 1] + cbytes, 0, 0, 0);
#endif
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
            const int off = pp * PAIR_B + (v * FH + u) * 4;
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
#pragma unroll 4
            for (int ch = 0; ch < 32; ++ch) {
                const int e = ch * RP + p;
                yo[(size_t)ch * hw + p] = ((S[e] + S[e + RW]) + S[e + 2 * RW]) + S[e + 3 * RW];
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
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int ch = (r >> 2) * 8 + slot * 4 + (r & 3);
                    const float v = acc[b][r] + R[ch * RP + p];
                    if (p < tile.npix) yo[(size_t)ch * hw + p] = v;
                }
            }
        }
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

template <int FH, int FW, int NB, int KS>
void launch_band_nb(const F32BandArgs& a, int64_t lds, hipStream_t stream) {
    if (a.mode == kBandGather)
        launch_band_v<FH, FW, NB, kBandGather, KS>(a, lds, stream);
    else if (a.mode == kBandNarrow)
        launch_band_v<FH, FW, NB, kBandNarrow, KS>(a, lds, stream);
    else
        launch_band_v<FH, FW, NB, kBandWide, KS>(a, lds, stream);
}

// Pixel blocks per band that the kernels are built for.
constexpr int kBandNb4Min = 4, kBandNb4Max = 7;     // four-way split
constexpr int kBandNb2Min = 12, kBandNb2Max = 13;   // two-way split (3x3)

constexpr int kBandMaxRounds = 4;   // rounds of 256 workgroups

bool band_shape_ok(const Geometry& g, int ks, int nb) {
    if (ks == 4) return nb >= kBandNb4Min && nb <= kBandNb4Max && g.fh == 3 && (g.fw == 3 || g.fw == 5);
    return nb >= kBandNb2Min && nb <= kBandNb2Max && g.fh == 3 && g.fw == 3 && g.k % 64 == 0;
}

}  // namespace

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
            if (rounds > kBandMaxRounds) continue;
            const double eff = useful / ((double)rounds * 1024.0 * nb * pp);
            if (eff > best.eff + 1e-9) {
                best.ks = ks;
                best.rows = (int)rows;
                best.nb = (int)nb;
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
    a.c = (int)g.c; a.h = (int)g.h; a.w = (int)g.w; a.k = (int)g.k;
    a.sh = (int)g.sh; a.sw = (int)g.sw; a.ph = (int)g.ph; a.pw = (int)g.pw;
    a.ho = (int)g.ho; a.wo = (int)g.wo;
    a.row_len = (int)g.row_len;
    a.div_row = make_fastdiv((uint32_t)g.row_len);
    a.div_wo = make_fastdiv((uint32_t)g.wo);
    a.plane_src = fused ? (int)(g.h * g.w) : (int)(g.ho * g.row_len);
    a.rows = p.rows;
    a.nbands = (int)((g.ho + p.rows - 1) / p.rows);
    a.ks = p.ks;
    a.nkt = (int)(g.k / (32 * (4 / p.ks)));
    a.nchunks = (int)(g.c / kBandChunk);
    a.grid = (int)p.grid;
    a.xcd_remap = (p.grid % 8 == 0 && p.grid > 8) ? 1 : 0;
    // 16-byte copies need 16-byte aligned planes
    const bool aligned = ((uintptr_t)src & 15) == 0 && (g.ho * g.row_len) % 4 == 0;
    a.mode = fused ? kBandGather : aligned ? kBandWide : kBandNarrow;
    return a;
}

int launch_conv_f32_band(const Geometry& g, const F32BandPlan& p, bool fused, const void* src, const void* w,
                         float* y, hipStream_t stream) {
    const F32BandArgs a = band_args_f32(g, p, fused, src, w, y);
    const int64_t lds = p.lds_bytes;
    if (p.ks == 2) {
        if (p.nb == 12) launch_band_nb<3, 3, 12, 2>(a, lds, stream);
        else launch_band_nb<3, 3, 13, 2>(a, lds, stream);
        return 0;
    }
#define BAND_NB4(FW_)                                                   \
    switch (p.nb) {                                                     \
        case 4: launch_band_nb<3, FW_, 4, 4>(a, lds, stream); break;    \
        case 5: launch_band_nb<3, FW_, 5, 4>(a, lds, stream); break;    \
        case 6: launch_band_nb<3, FW_, 6, 4>(a, lds, stream); break;    \
        default: launch_band_nb<3, FW_, 7, 4>(a, lds, stream); break;   \
    }
    if (g.fw == 3) {
        BAND_NB4(3)
    } else {
        BAND_NB4(5)
    }
#undef BAND_NB4
    return 0;
}

}  // namespace im2win
