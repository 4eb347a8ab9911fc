// bf16 im2win convolution with one image per workgroup (small feature maps:
// a whole image's window strips of a 32-channel chunk fit in LDS).
//
// The same implicit GEMM as the other convolution kernels (Alg. 2: the
// window of output pixel (m, n) is the run [n*sw*Fh, (n*sw + Fw)*Fh) of
// window-tensor row m; tap (u, v) sits at offset v*Fh + u), with the work cut
// so that a feature map of a few hundred pixels fills the chip evenly:
//   - a workgroup owns one image and 128 output channels (grid N * K/128); each
//     of its 8 waves computes 32 output channels (2 blocks of 16) for half of
//     the image's pixels (NPB blocks of 16), with v_mfma_f32_16x16x32_bf16
//     and fp32 accumulation.  Waves w and w + 4 share a SIMD and split one
//     image's pixels for the same 32 channels, so every SIMD does the same
//     work, and each SIMD has a second wave to issue while one waits;
//   - the reduction runs over chunks of 32 input channels; one MFMA contracts
//     the 32 channels of one tap, 8 consecutive channels per lane group of 16;
//   - window strips go through LDS channel-innermost (4 planes of 8 channels,
//     16 bytes per position), one image's rows per chunk, in two stages;
//     each B fragment is one 16-byte LDS read per lane, the taps of a window
//     being immediate offsets from the pixel's window start.  The row pitch
//     is congruent to sw*Fh*Wo modulo 16 positions, so the windows of 16
//     consecutive pixels start in 16 different bank groups when sw*Fh is odd;
//   - the filter does not go through LDS: pack_filter_frag_kernel rewrites it
//     into the caller's scratch in MFMA-fragment order, and each wave loads
//     its two fragments of a tap straight into registers with one 16-byte
//     load per lane each, a whole chunk ahead;
//   - unfused, the strips are the window-tensor rows of the image (8-byte
//     loads of 4 positions of 8 channels, transposed in registers); fused,
//     pairs of input elements of 8 channels are transposed and written to
//     every window row that holds them (the transform's scatter, on chip),
//     and the padding positions stay zero from a clear at the start.
// Workgroups of one image are placed on the same XCD (the hardware hands
// consecutive workgroup ids to the 8 XCDs in turn), so they share the image
// in that XCD's L2.
#include "conv_common.h"

#include <cstdio>

namespace im2win {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ inline uint32_t lo_pair(uint32_t a, uint32_t b) { return (a & 0xffffu) | (b << 16); }
__device__ inline uint32_t hi_pair(uint32_t a, uint32_t b) { return (a >> 16) | (b & 0xffff0000u); }

// Raw buffer resource over `bytes` bytes at p (loads past the end read 0).
__device__ inline __amdgpu_buffer_rsrc_t buffer_rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

// Scheduling fences: every instruction kind but global/buffer memory
// accesses may cross them, so the loads stay where they are issued (the
// compiler would otherwise sink them next to their first use, which
// exposes their whole latency) while LDS reads and MFMAs still interleave.
#define IMG_PIN_VMEM() __builtin_amdgcn_sched_barrier(0x0001 | 0x0002 | 0x0004 | 0x0008 | 0x0080 | 0x0100 | 0x0200)

template <int FH, int FW, bool FUSED, int NPB>
__global__ __launch_bounds__(kImgThreads, 1) void conv_bf16_image_kernel(ImgArgs a) {
    constexpr int T = FH * FW;
    constexpr int SI = FUSED ? kImgFusedItems : kImgStripItems;   // staging items per thread
    extern __shared__ __align__(16) unsigned char smem[];
    u32x4* L = reinterpret_cast<u32x4*>(smem);   // 16-byte positions

    const int tid = threadIdx.x, lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform (scalar registers)
    const int kp = wv & 3, half = wv >> 2;   // 32 output channels, half of the pixel blocks
    const int bid = a.xcd_remap ? (int)(blockIdx.x & 7) * (a.grid >> 3) + (int)(blockIdx.x >> 3)
                                : (int)blockIdx.x;
    const int img = bid / a.nkt, kt = bid - img * a.nkt;
    const int g = lane >> 4;   // channel group of this lane's 8 reduction elements

    // Window start (position, in this lane's channel plane) of the lane's
    // pixel in each pixel block; pixels past the image are clamped to its
    // last pixel (computed, never stored).
    int posb[NPB];
#pragma unroll
    for (int q = 0; q < NPB; ++q) {
        int p = (half * NPB + q) * 16 + (lane & 15);
        if (p > a.npix - 1) p = a.npix - 1;
        const int m = p / a.wo, n = p - m * a.wo;
        posb[q] = g * a.plane_pos + m * a.pitch + n * a.sw * FH;
    }

    // Filter fragments of this wave: pair kp of 16-channel blocks (32 output
    // channels), chunk ch, tap t, block i at fragment ((kp*nchunks + ch)*T +
    // t)*2 + i, 1 KB each (16 bytes per lane).
    const __amdgpu_buffer_rsrc_t wres = buffer_rsrc(a.wf, (uint32_t)a.k * a.c * T * 2);
    const int wlane = lane * 16;
    const int wq0 = (kt * 4 + kp) * a.nchunks * T * 2 * 1024;

    // Staging items, the same every chunk: (channel group, 4 positions) of
    // the window tensor, or (channel group, 2 input elements) of x.  A thread
    // beyond the last item repeats the item of its lane in the first wave
    // (the same loads, the same values to the same positions), so the
    // staging has no branch.
    int src_off[SI];               // byte offset from channel 8*group of the chunk's first channel
    int dst[SI][FUSED ? FH : 1];   // LDS position (-1: none)
    int odd_ok[SI];                // fused: the second element of the pair lands in the rows too
    {
        const int nitems = 4 * a.ngroups;
#pragma unroll
        for (int k = 0; k < SI; ++k) {
            int item = tid + k * kImgThreads;
            if (item >= nitems) item = lane < nitems ? lane : 0;
            const int gg = item / a.ngroups, e = item - gg * a.ngroups;
            odd_ok[k] = 0;
            if constexpr (!FUSED) {
                src_off[k] = (gg * 8 * a.plane_src + 4 * e) * 2;
                const int m = (4 * e) / a.row_len, q = 4 * e - m * a.row_len;
                dst[k][0] = gg * a.plane_pos + m * a.pitch + q;
            } else {
                src_off[k] = (gg * 8 * a.plane_src + 2 * e) * 2;
                const int yy = (2 * e) / a.w, xx = 2 * e - yy * a.w;
#pragma unroll
                for (int u = 0; u < FH; ++u) {
                    const int t = yy + a.ph - u;
                    const int m = t >= 0 ? t / a.sh : -1;
                    const bool hit = t >= 0 && m * a.sh == t && m < a.ho && xx + a.pw < a.wr;
                    dst[k][u] = hit ? gg * a.plane_pos + m * a.pitch + (xx + a.pw) * FH + u : -1;
                }
                odd_ok[k] = xx + 1 + a.pw < a.wr ? 1 : 0;
            }
        }
    }

    const size_t img_elems = (size_t)a.c * a.plane_src;
    const __amdgpu_buffer_rsrc_t sres = buffer_rsrc(a.src + (size_t)img * img_elems, (uint32_t)(img_elems * 2));
    const int plane_bytes = a.plane_src * 2;
    uint32_t sr[SI][FUSED ? 8 : 16];

    auto load_strips = [&](int ch) {
        const int cbase = ch * kImgChunk * plane_bytes;
#pragma unroll
        for (int k = 0; k < SI; ++k) {
#pragma unroll
            for (int c8 = 0; c8 < 8; ++c8) {
                if constexpr (!FUSED) {
                    const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(sres, src_off[k], cbase + c8 * plane_bytes, 0);
                    sr[k][2 * c8] = v[0];
                    sr[k][2 * c8 + 1] = v[1];
                } else {
                    sr[k][c8] = __builtin_amdgcn_raw_buffer_load_b32(sres, src_off[k], cbase + c8 * plane_bytes, 0);
                }
            }
        }
    };
    auto store_strips = [&](int stage) {
        u32x4* S = L + stage * a.stage_pos;
#pragma unroll
        for (int k = 0; k < SI; ++k) {
            if constexpr (!FUSED) {
                // The 16 lanes of a store cover 16 consecutive groups of 4
                // positions; writing position r = (pq + dst/16) mod 4 of its
                // group in store pq puts them in 16 different bank groups.
                // Word e of position r holds channels 2e, 2e+1: the low or
                // high halves (r odd) of the words of positions r & 2.
                const int rot = dst[k][0] >> 4;
#pragma unroll
                for (int pq = 0; pq < 4; ++pq) {
                    const int r = (pq + rot) & 3;
                    const uint32_t sel = (r & 1) ? 0x07060302u : 0x05040100u;
                    const bool upper = (r & 2) != 0;
                    u32x4 o;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const uint32_t w0 = upper ? sr[k][4 * e + 1] : sr[k][4 * e];
                        const uint32_t w1 = upper ? sr[k][4 * e + 3] : sr[k][4 * e + 2];
                        o[e] = __builtin_amdgcn_perm(w1, w0, sel);
                    }
                    S[dst[k][0] + r] = o;
                }
            } else {
                u32x4 o0, o1;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    o0[e] = lo_pair(sr[k][2 * e], sr[k][2 * e + 1]);
                    o1[e] = hi_pair(sr[k][2 * e], sr[k][2 * e + 1]);
                }
#pragma unroll
                for (int u = 0; u < FH; ++u) {
                    if (dst[k][u] >= 0) {
                        S[dst[k][u]] = o0;
                        if (odd_ok[k]) S[dst[k][u] + FH] = o1;
                    }
                }
            }
        }
    };

    if constexpr (FUSED) {
        // padding positions are never written by the scatter: clear both stages
        const u32x4 z = {0u, 0u, 0u, 0u};
        for (int i = tid; i < 2 * a.stage_pos; i += kImgThreads) L[i] = z;
        __syncthreads();
    }

    f32x4 acc[2][NPB];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int q = 0; q < NPB; ++q) acc[i][q] = f32x4{0.f, 0.f, 0.f, 0.f};

    // A fragments of the current chunk, by tap.  The loads of the next
    // chunk's tap t are issued right after the MFMAs of tap t, so each has a
    // whole chunk to arrive; they follow the strip loads of the next chunk in
    // issue order, and those are waited for (at the end of this chunk)
    // before any of them is needed.
    u32x4 af[T][2];
#pragma unroll
    for (int t = 0; t < T; ++t)
#pragma unroll
        for (int i = 0; i < 2; ++i) af[t][i] = __builtin_amdgcn_raw_buffer_load_b128(wres, wlane, wq0 + (t * 2 + i) * 1024, 0);
    load_strips(0);
    store_strips(0);
    __syncthreads();

    // Every chunk but the last: the next chunk's strips and filter are loaded
    // while this one is multiplied.
    for (int ch = 0; ch + 1 < a.nchunks; ++ch) {
        const int nx = ch + 1;
        IMG_PIN_VMEM();
        load_strips(nx);
        IMG_PIN_VMEM();
        const u32x4* S = L + (ch & 1) * a.stage_pos;
        const int wn = wq0 + nx * T * 2 * 1024;
        // B fragments stream through a ring of kImgBRing registers, read
        // kImgBRing - 1 steps ahead of the two MFMAs that use them (steps run
        // over taps, then pixel blocks); one LDS read and two MFMAs per step.
        constexpr int NS = T * NPB, R = kImgBRing;
        u32x4 bq[R];
#pragma unroll
        for (int s0 = 0; s0 < R - 1; ++s0) bq[s0] = S[posb[s0 % NPB] + s0 / NPB];
#pragma unroll
        for (int st = 0; st < NS; ++st) {
            const int t = st / NPB, q = st % NPB;
            if (st + R - 1 < NS) {
                const int s1 = st + R - 1;
                bq[s1 % R] = S[posb[s1 % NPB] + s1 / NPB];
            }
            // nothing crosses: the read stays R - 1 steps ahead of its use
            // (the compiler would sink it next to its MFMAs)
            __builtin_amdgcn_sched_barrier(0);
            const bf16x8 bv = __builtin_bit_cast(bf16x8, bq[st % R]);
#pragma unroll
            for (int i = 0; i < 2; ++i)
                acc[i][q] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, af[t][i]), bv,
                                                                    acc[i][q], 0, 0, 0);
            if (q == NPB - 1) {
                IMG_PIN_VMEM();
#pragma unroll
                for (int i = 0; i < 2; ++i)
                    af[t][i] = __builtin_amdgcn_raw_buffer_load_b128(wres, wlane, wn + (t * 2 + i) * 1024, 0);
                IMG_PIN_VMEM();
            }
        }
        store_strips((ch + 1) & 1);
        __syncthreads();
    }

    // The last chunk runs pixel block by pixel block (taps inner), and each
    // block's outputs are stored as soon as its last MFMAs are issued, so
    // the stores of the first blocks drain while the later ones multiply.
    // D[row][col]: col = lane % 16 (pixel), row = 4*(lane/16) + v (output
    // channel).
    float* yimg = a.y + (size_t)img * a.k * a.npix;
    {
        const u32x4* S = L + ((a.nchunks - 1) & 1) * a.stage_pos;
        constexpr int NS = T * NPB, R = kImgBRing;
        u32x4 bq[R];
#pragma unroll
        for (int s0 = 0; s0 < R - 1; ++s0) bq[s0] = S[posb[s0 / T] + s0 % T];
#pragma unroll
        for (int st = 0; st < NS; ++st) {
            const int q = st / T, t = st % T;
            if (st + R - 1 < NS) {
                const int s1 = st + R - 1;
                bq[s1 % R] = S[posb[s1 / T] + s1 % T];
            }
            __builtin_amdgcn_sched_barrier(0);
            const bf16x8 bv = __builtin_bit_cast(bf16x8, bq[st % R]);
#pragma unroll
            for (int i = 0; i < 2; ++i)
                acc[i][q] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, af[t][i]), bv,
                                                                    acc[i][q], 0, 0, 0);
            if (t == T - 1) {
                const int p = (half * NPB + q) * 16 + (lane & 15);
                if (p < a.npix) {
#pragma unroll
                    for (int i = 0; i < 2; ++i)
#pragma unroll
                        for (int v = 0; v < 4; ++v) {
                            const int j = kt * 128 + kp * 32 + i * 16 + 4 * g + v;
                            yimg[(size_t)j * a.npix + p] = acc[i][q][v];
                        }
                }
            }
        }
    }
}

// The filter K x C x Fh x Fw rewritten in fragment order: fragment
// ((kp*nchunks + ch)*T + t)*2 + i holds, for lane l, the 8 channels
// 32*ch + 8*(l/16) .. +7 of tap t = v*Fh + u of output channel
// 32*kp + 16*i + l%16, as one 16-byte piece.  One wave per (16 output
// channels, chunk): each lane loads the contiguous run of its output
// channel's 8 channels x T taps (16*T bytes, T 16-byte loads, all in flight
// at once), picks each tap's 8 values out of it with byte permutes and
// stores the T pieces; a store instruction writes one whole fragment.
template <int FH, int FW>
__global__ __launch_bounds__(64) void pack_filter_frag_kernel(const uint16_t* __restrict__ w,
                                                              uint16_t* __restrict__ wf, int c, int nchunks) {
    constexpr int T = FH * FW;
    const int lane = threadIdx.x;
    const int ch = (int)blockIdx.x % nchunks, kb = (int)blockIdx.x / nchunks;   // kb: block of 16 output channels
    const int k = kb * 16 + (lane & 15), g = lane >> 4;
    const u32x4* run = reinterpret_cast<const u32x4*>(w + ((size_t)k * c + kImgChunk * ch + 8 * g) * T);
    uint32_t d[4 * T];   // run element e (channel e / T, natural tap e % T) in half e & 1 of word e / 2
#pragma unroll
    for (int q = 0; q < T; ++q) {
        const u32x4 v = run[q];
#pragma unroll
        for (int e = 0; e < 4; ++e) d[4 * q + e] = v[e];
    }
    const int kp = kb >> 1, i = kb & 1;
    u32x4* out = reinterpret_cast<u32x4*>(wf) + (((size_t)kp * nchunks + ch) * T * 2 + i) * 64 + lane;
#pragma unroll
    for (int t = 0; t < T; ++t) {
        const int vv = t / FH, u = t - vv * FH, nat = u * FW + vv;
        u32x4 o;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int e0 = (2 * j) * T + nat, e1 = (2 * j + 1) * T + nat;
            // bytes 0-1: half e0 & 1 of word e0 / 2 (second operand); bytes
            // 2-3: half e1 & 1 of word e1 / 2 (first operand, selectors 4-7)
            const uint32_t sel = (uint32_t)((e0 & 1) * 2) | (uint32_t)((e0 & 1) * 2 + 1) << 8 |
                                 (uint32_t)(4 + (e1 & 1) * 2) << 16 | (uint32_t)(4 + (e1 & 1) * 2 + 1) << 24;
            o[j] = __builtin_amdgcn_perm(d[e1 >> 1], d[e0 >> 1], sel);
        }
        out[(size_t)t * 2 * 64] = o;
    }
}

template <int FH, int FW, int NPB>
void launch_image(const ImgArgs& a, bool fused, int64_t lds, hipStream_t stream) {
    auto kern = fused ? conv_bf16_image_kernel<FH, FW, true, NPB> : conv_bf16_image_kernel<FH, FW, false, NPB>;
    if (lds > 64 * 1024)
        (void)hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL(kern, dim3((unsigned)a.grid), dim3(kImgThreads), (size_t)lds, stream, a);
}

}  // namespace

ImgPlan plan_image_bf16(const Geometry& g, bool fused) {
    ImgPlan p;
    if (g.elem != 2 || g.fh != 3 || g.fw != 3) return p;
    if (g.c % kImgChunk || g.k % 128 || g.k > 1024) return p;
    const int64_t npix = g.ho * g.wo;
    const int64_t nblk = (npix + 15) / 16;
    if (nblk > 2 * kImgNPB || nblk < 2 * kImgNPB - 2) return p;   // the kernel's 2 x NPB pixel blocks
    if ((g.sw * g.fh) % 2 == 0) return p;                         // bank-conflict-free windows
    // both variants or neither: 16-byte-aligned groups of 4 window-tensor
    // positions, pairs of input elements, each within the staging registers
    if (g.w % 2 != 0 || g.row_len % 4 != 0) return p;
    if (g.ho * g.row_len > (int64_t)kImgStripItems * kImgThreads ||
        2 * g.h * g.w > (int64_t)kImgFusedItems * kImgThreads)
        return p;
    const int64_t pitch = g.row_len + mod16((int)((g.sw * g.fh * g.wo - g.row_len) % 16));
    // planes start on multiples of 16 positions: the four 16-lane groups of
    // a fragment read then run at full LDS rate (measured on this GPU: any
    // other plane offset modulo 16 costs a third of the read bandwidth)
    const int64_t ext = g.ho * pitch + 16;
    const int64_t plane_pos = (ext + 15) & ~int64_t(15);
    const int64_t stage_pos = 4 * plane_pos;
    const int64_t lds = 2 * stage_pos * 16;
    if (lds > kConvLdsMaxBytes) return p;
    const int64_t plane_src = fused ? g.h * g.w : g.ho * g.row_len;
    const int64_t ngroups = fused ? plane_src / 2 : plane_src / 4;
    const int64_t grid = g.n * (g.k / 128);
    if (grid > 0x7fffffff || g.n * g.c * g.h * g.w >= (int64_t(1) << 31) ||
        g.n * g.c * g.ho * g.row_len >= (int64_t(1) << 31) ||
        g.n * g.k * npix >= (int64_t(1) << 31))
        return p;
    p.ok = true;
    p.pitch = pitch;
    p.plane_pos = plane_pos;
    p.stage_pos = stage_pos;
    p.lds_bytes = lds;
    p.plane_src = plane_src;
    p.ngroups = ngroups;
    p.grid = grid;
    return p;
}

ImgArgs image_args(const Geometry& g, const ImgPlan& p, const void* src, const void* wf, float* y) {
    ImgArgs a;
    a.src = static_cast<const uint16_t*>(src);
    a.wf = static_cast<const uint16_t*>(wf);
    a.y = y;
    a.c = (int)g.c; a.h = (int)g.h; a.w = (int)g.w; a.k = (int)g.k;
    a.sh = (int)g.sh; a.sw = (int)g.sw; a.ph = (int)g.ph; a.pw = (int)g.pw;
    a.ho = (int)g.ho; a.wo = (int)g.wo; a.wr = (int)g.wp; a.row_len = (int)g.row_len;
    a.npix = (int)(g.ho * g.wo);
    a.pitch = (int)p.pitch;
    a.plane_pos = (int)p.plane_pos;
    a.stage_pos = (int)p.stage_pos;
    a.plane_src = (int)p.plane_src;
    a.ngroups = (int)p.ngroups;
    a.nkt = (int)(g.k / 128);
    a.nchunks = (int)(g.c / kImgChunk);
    a.grid = (int)p.grid;
    a.xcd_remap = (p.grid % 8 == 0 && a.nkt > 1) ? 1 : 0;
    return a;
}

int launch_conv_bf16_image(const Geometry& g, const ImgPlan& p, bool fused, const void* src,
                           const void* w, void* scratch, float* y, hipStream_t stream) {
    const int nchunks = (int)(g.c / kImgChunk);
    hipLaunchKernelGGL((pack_filter_frag_kernel<3, 3>), dim3((unsigned)(g.k / 16 * nchunks)), dim3(64), 0, stream,
                       static_cast<const uint16_t*>(w), static_cast<uint16_t*>(scratch), (int)g.c, nchunks);
    const ImgArgs a = image_args(g, p, src, scratch, y);
    launch_image<3, 3, kImgNPB>(a, fused, p.lds_bytes, stream);
    return 0;
}

}  // namespace im2win
