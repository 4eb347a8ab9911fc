// fp32 im2win convolution with one image per workgroup (small feature maps:
// the window strips of one image fit in LDS a few channels at a time).
//
// The same implicit GEMM as the other convolution kernels (Alg. 2: the
// window of output pixel (m, n) is the run [n*sw*Fh, (n*sw + Fw)*Fh) of
// window-tensor row m; tap (u, v) sits at offset v*Fh + u), cut so that a
// feature map of 100 to 224 pixels fills the chip without tile quantization:
//   - a workgroup owns one image and 32 output channels (grid N * K/32) and
//     computes all of the image's pixels, NB blocks of 32, with
//     v_mfma_f32_32x32x2f32 (A = 32 filter rows, B = 32 pixel windows);
//   - the reduction runs over chunks of 8 input channels; each of the 4
//     waves takes 2 of them (one per k-slot of the matrix core) through all
//     Fh*Fw taps, so the waves split the reduction evenly and every SIMD
//     does the same work; the four partial sums are added in a fixed order
//     through LDS at the end;
//   - a chunk's strips sit in LDS in the window tensor's own layout (one
//     slot of Ho*L elements per channel), two chunks deep.  Unfused, each
//     channel's strip is one contiguous run of the window tensor, copied by
//     LDS DMA (buffer_load ... lds, no register round trip) in 16-byte
//     pieces, or 4-byte ones when Ho*L is not a multiple of 4.  Fused, every
//     strip element is gathered from x by 4-byte LDS DMA with per-lane source
//     offsets computed once per kernel; padding positions carry an offset
//     past the end of the buffer, which the hardware reads as zero;
//   - the filter does not go through LDS: each lane loads its own filter row
//     (one output channel, one input channel, Fh*Fw taps) of the next chunk
//     into registers while the current chunk is multiplied.
// Both variants stage the same values into the same positions and run the
// same matrix-core sequence, so their outputs are bitwise identical.
// Workgroups of one image are placed on the same XCD (the hardware hands
// consecutive workgroup ids to the 8 XCDs in turn), so they share the image
// in that XCD's L2.
#include "conv_common.h"

#include <cstdio>
#include <type_traits>

namespace im2win {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void;

// Raw buffer resource over `bytes` bytes at p (loads past the end read 0).
__device__ inline __amdgpu_buffer_rsrc_t buffer_rsrc_f32(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

// Scheduling fence that keeps global/buffer memory accesses where they are
// issued while LDS reads and MFMAs may still interleave across it.
#define F32IMG_PIN_VMEM() __builtin_amdgcn_sched_barrier(0x0001 | 0x0002 | 0x0004 | 0x0008 | 0x0080 | 0x0100 | 0x0200)

template <int FH, int FW, int NB, int MODE>
__global__ __launch_bounds__(kF32ImgThreads, 1) void conv_f32_image_kernel(F32ImgArgs a) {
    constexpr int T = FH * FW;
    constexpr int SC = kF32ImgSlot;                  // LDS floats per channel slot
    constexpr int STAGE_B = kF32ImgChunk * SC * 4;   // LDS bytes per stage
    constexpr int NJ = f32img_copies(MODE);          // copies per wave per chunk
    constexpr int NS = NJ / 2;                       // copies per channel slot
    constexpr int DPT = (NJ + T - 1) / T;            // copies issued after each tap
    extern __shared__ __align__(16) float S[];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform (scalar registers)
    const int bid = a.xcd_remap ? (int)(blockIdx.x & 7) * (a.grid >> 3) + (int)(blockIdx.x >> 3)
                                : (int)blockIdx.x;
    const int img = bid / a.nkt, kt = bid - img * a.nkt;
    const int slot = lane >> 5;     // k-slot: channel 2*wv + slot of every chunk
    const int col = lane & 31;      // A: output channel kt*32 + col; B: pixel b*32 + col

    // Window start (LDS byte address, stage 0) of the lane's pixel in each
    // pixel block, in its channel slot; pixels past the image are clamped to
    // its last pixel (computed, never stored).  Stage 1 and the tap are
    // immediate offsets of the read.
    uint32_t bb[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) bb[b] = f32img_window(a, FH, wv, lane, b);

    // Filter row of this lane: output channel kt*32 + col, input channel
    // ch*8 + 2*wv + slot, taps 0 .. T-1 (natural (u, v) order).
    const __amdgpu_buffer_rsrc_t wres = buffer_rsrc_f32(a.wt, (uint32_t)((size_t)a.k * a.c * T * 4));
    const int wlane = (((kt * 32 + col) * a.c) + 2 * wv + slot) * T * 4;

    // Source of the staging copies: the image's window-tensor planes, or the
    // image's input planes.
    const size_t img_elems = (size_t)a.c * a.plane_src;
    const __amdgpu_buffer_rsrc_t sres = buffer_rsrc_f32(a.src + (size_t)img * img_elems, (uint32_t)(img_elems * 4));
    const int plane_bytes = a.plane_src * 4;

    // Per-lane source byte offset (within one channel plane) of each copy of
    // a slot, the same for every channel and chunk (f32img_source).  Copies
    // past the strip or into the padding read from outside the buffer, which
    // yields zeros, so every copy is issued unconditionally and the slot's
    // tail beyond the strip is never read.
    uint32_t sofs[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) sofs[s] = f32img_source(a, MODE, FH, s, lane);

    // Copy j of chunk ch into stage ST: channel slot 2*wv + (j & 1), part
    // j >> 1.  A chunk past the last one reads only zeros (harmless: that
    // stage is not read again).
    auto copy = [&](int j, int ch, auto st_tag) {
        constexpr int ST = decltype(st_tag)::value;
        const uint32_t cbytes = (uint32_t)((ch * kF32ImgChunk + 2 * wv + (j & 1)) * plane_bytes);
        char* dst = reinterpret_cast<char*>(S) + ST * STAGE_B + f32img_dest(MODE, wv, j);
#if defined(__HIP_DEVICE_COMPILE__)   // (16-byte LDS copies exist on gfx950 only; the host pass checks them too)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(sres, (lds_void*)dst, MODE == kF32ImgWide ? 16 : 4, sofs[j >> 1] + cbytes, 0, 0, 0);
#endif
    };

    float fa0[T], fa1[T];
    auto load_filter_tap = [&](int ch, int t) {
        return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(wres, wlane + t * 4,
                                                                             ch * kF32ImgChunk * T * 4, 0));
    };

    f32x16 acc[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[b][r] = 0.0f;

    // One chunk from stage ST with filter registers fa, while the copies of
    // chunk ch + 1 into the other stage and its filter rows (into fn) are
    // issued between the taps.  The windows of tap t + 1 are read before the
    // MFMAs of tap t, so their LDS latency hides behind matrix-core work; the
    // scheduling fences keep the reads ahead of the copies, which the
    // compiler cannot tell apart from the stage being read.
    auto chunk = [&](auto st_tag, const float (&fa)[T], float (&fn)[T], int ch) {
        constexpr int ST = decltype(st_tag)::value;
        const char* base = reinterpret_cast<const char*>(S) + ST * STAGE_B;
        float bv[2][NB];
        auto read_tap = [&](int t, float (&dst)[NB]) {
            const int u = t / FW, v = t - u * FW;
            const int toff = (v * FH + u) * 4;
#pragma unroll
            for (int b = 0; b < NB; ++b) dst[b] = *reinterpret_cast<const float*>(base + bb[b] + toff);
        };
        read_tap(0, bv[0]);
#pragma unroll
        for (int t = 0; t < T; ++t) {
            if (t + 1 < T) read_tap(t + 1, bv[(t + 1) & 1]);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int b = 0; b < NB; ++b)
                acc[b] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[t], bv[t & 1][b], acc[b], 0, 0, 0);
            F32IMG_PIN_VMEM();
#pragma unroll
            for (int d = 0; d < DPT; ++d)
                if (t * DPT + d < NJ) copy(t * DPT + d, ch + 1, std::integral_constant<int, 1 - ST>());
            fn[t] = load_filter_tap(ch + 1, t);
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
    for (int t = 0; t < T; ++t) fa0[t] = load_filter_tap(0, t);
    land();
    for (int ch = 0; ch < a.nchunks; ch += 2) {   // nchunks is even
        chunk(std::integral_constant<int, 0>(), fa0, fa1, ch);
        land();
        chunk(std::integral_constant<int, 1>(), fa1, fa0, ch + 1);
        land();
    }

    // Partial sums of the four waves: R[wave][channel][pixel] in LDS, then
    // y = ((R0 + R1) + R2) + R3, one pixel per thread, 32 channels each.
    constexpr int RP = NB * 32;
    float* R = S;
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int ch = (r >> 2) * 8 + slot * 4 + (r & 3);
            R[(wv * 32 + ch) * RP + b * 32 + col] = acc[b][r];
        }
    __syncthreads();
    if (tid < a.npix) {
        float* yo = a.y + ((size_t)img * a.k + (size_t)kt * 32) * a.npix + tid;
        constexpr int RW = 32 * RP;
#pragma unroll 4
        for (int ch = 0; ch < 32; ++ch) {
            const int e = ch * RP + tid;
            yo[(size_t)ch * a.npix] = ((R[e] + R[e + RW]) + R[e + 2 * RW]) + R[e + 3 * RW];
        }
    }
}

template <int FH, int FW, int NB, int MODE>
void launch_f32_image_v(const F32ImgArgs& a, int64_t lds, hipStream_t stream) {
    if (lds > 64 * 1024)
        (void)hipFuncSetAttribute((const void*)conv_f32_image_kernel<FH, FW, NB, MODE>,
                                  hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL((conv_f32_image_kernel<FH, FW, NB, MODE>), dim3((unsigned)a.grid), dim3(kF32ImgThreads),
                       (size_t)lds, stream, a);
}

template <int FH, int FW, int NB>
void launch_f32_image_nb(const F32ImgArgs& a, int64_t lds, hipStream_t stream) {
    if (a.mode == kF32ImgGather)
        launch_f32_image_v<FH, FW, NB, kF32ImgGather>(a, lds, stream);
    else if (a.mode == kF32ImgNarrow)
        launch_f32_image_v<FH, FW, NB, kF32ImgNarrow>(a, lds, stream);
    else
        launch_f32_image_v<FH, FW, NB, kF32ImgWide>(a, lds, stream);
}

template <int FH, int FW>
void launch_f32_image_f(const F32ImgArgs& a, int nb, int64_t lds, hipStream_t stream) {
    switch (nb) {
        case 4: launch_f32_image_nb<FH, FW, 4>(a, lds, stream); break;
        case 5: launch_f32_image_nb<FH, FW, 5>(a, lds, stream); break;
        case 6: launch_f32_image_nb<FH, FW, 6>(a, lds, stream); break;
        default: launch_f32_image_nb<FH, FW, 7>(a, lds, stream); break;
    }
}

}  // namespace

F32ImgPlan plan_image_f32(const Geometry& g) {
    F32ImgPlan p;
    if (g.elem != 4 || g.fh != 3 || (g.fw != 3 && g.fw != 5)) return p;
    if (g.c % (2 * kF32ImgChunk) || g.k % 32) return p;
    const int64_t npix = g.ho * g.wo;
    const int64_t nb = (npix + 31) / 32;
    if (nb < kF32ImgMinNB || nb > kF32ImgMaxNB) return p;
    const int64_t grid = g.n * (g.k / 32);
    if (grid < 256) return p;   // fewer workgroups than compute units: the tiled kernels spread wider
    const int64_t plane_strip = g.ho * g.row_len;
    if (plane_strip > 64 * kF32ImgMaxSeg) return p;
    const int64_t lds = std::max<int64_t>(2 * kF32ImgChunk * kF32ImgSlot * 4, 4 * 32 * nb * 32 * 4);
    if (lds > kConvLdsMaxBytes) return p;
    // 32-bit buffer offsets, with the out-of-buffer offset beyond every slab
    // (x or window tensor of one image) and every chunk index
    if (g.c * g.h * g.w * 4 >= (int64_t(1) << 30) || g.c * plane_strip * 4 >= (int64_t(1) << 30) ||
        g.k * g.c * g.taps * 4 >= (int64_t(1) << 31) || g.n * g.k * npix >= (int64_t(1) << 31) ||
        grid > 0x7fffffff)
        return p;
    p.ok = true;
    p.nb = (int)nb;
    p.lds_bytes = lds;
    p.grid = grid;
    return p;
}

F32ImgArgs image_args_f32(const Geometry& g, const F32ImgPlan& p, bool fused, const void* src, const void* w,
                          float* y) {
    F32ImgArgs a;
    a.src = static_cast<const float*>(src);
    a.wt = static_cast<const float*>(w);
    a.y = y;
    a.c = (int)g.c; a.h = (int)g.h; a.w = (int)g.w; a.k = (int)g.k;
    a.sh = (int)g.sh; a.sw = (int)g.sw; a.ph = (int)g.ph; a.pw = (int)g.pw;
    a.ho = (int)g.ho; a.wo = (int)g.wo;
    a.row_len = (int)g.row_len;
    a.div_row = make_fastdiv((uint32_t)g.row_len);
    a.div_wo = make_fastdiv((uint32_t)g.wo);
    a.npix = (int)(g.ho * g.wo);
    a.plane_strip = (int)(g.ho * g.row_len);
    a.plane_src = fused ? (int)(g.h * g.w) : a.plane_strip;
    a.nkt = (int)(g.k / 32);
    a.nchunks = (int)(g.c / kF32ImgChunk);
    a.grid = (int)p.grid;
    a.xcd_remap = (p.grid % 8 == 0 && a.nkt > 1) ? 1 : 0;
    a.mode = fused ? kF32ImgGather : (a.plane_strip % 4 == 0 ? kF32ImgWide : kF32ImgNarrow);
    return a;
}

int launch_conv_f32_image(const Geometry& g, const F32ImgPlan& p, bool fused, const void* src, const void* w,
                          float* y, hipStream_t stream) {
    const F32ImgArgs a = image_args_f32(g, p, fused, src, w, y);
    if (g.fw == 3)
        launch_f32_image_f<3, 3>(a, p.nb, p.lds_bytes, stream);
    else
        launch_f32_image_f<3, 5>(a, p.nb, p.lds_bytes, stream);
    return 0;
}

}  // namespace im2win
