// bf16 im2win convolution on gfx950 matrix cores, fp32 accumulation.
//
// Same implicit GEMM and pixel tiling as the fp32 kernel (Alg. 2 semantics),
// with the reduction ordered tap-major inside a chunk of 16 input channels:
// kk = (t, r), t = v*Fh + u.  v_mfma_f32_32x32x16_bf16 contracts the 16
// channels of one tap per instruction (8 consecutive reduction elements per
// lane), so the LDS holds the window strips channel-innermost, S[pos][16]: a
// lane's B operand for pixel p and tap t is the 16-byte vector
// S[base(p) + t][8h .. 8h+7].  A strip position is still the window-tensor
// element at that row position, so the window of a pixel stays the contiguous
// run of positions [base(p), base(p) + Fw*Fh), shared with the overlapping
// windows of its neighbours (Sec. III-B).  The filter is held as F[t][j][16].
//
// Neither operand has that layout in memory (the window tensor and the filter
// are channel-outer), so each chunk passes through registers:
//   - right after the barrier that opens chunk c, every thread loads its
//     items of chunk c+1: 16-byte loads of 8 strip positions for each of 8
//     channels, and of one output channel's filter row for 8 channels and all
//     taps; they land while the MFMAs of chunk c run;
//   - after those MFMAs the items are transposed in registers (16-bit lane
//     permutes) and written to the other of two LDS stages with 16-byte
//     stores, so one barrier per chunk suffices.
// The fused kernel gathers the strip positions from x (zero in the padding)
// with 2-byte loads, as do shapes whose window-tensor planes or filter rows
// are not whole 16-byte vectors.  Channels beyond C are zero in both
// operands.
#include "conv_common.h"

#include <cstdio>

namespace im2win {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kRC = kBf16Chunk;                            // channels per chunk (MFMA reduction width)
constexpr int kStripVecItems = kBf16StripVecItems;         // 8 positions x 8 channels, 16-byte loads
constexpr int kStripScalarItems = kBf16StripScalarItems;   // 1 position x 8 channels, 2-byte loads
constexpr int kFilterScalarItems = kBf16FilterScalarItems; // 1 tap x 8 channels, 2-byte loads

enum StripMode { kStripVec = 0, kStripScalar = 1, kStripFused = 2 };

// (lo16(a), lo16(b)) and (hi16(a), hi16(b)) as one 32-bit word
__device__ inline uint32_t lo_pair(uint32_t a, uint32_t b) { return (a & 0xffffu) | (b << 16); }
__device__ inline uint32_t hi_pair(uint32_t a, uint32_t b) { return (a >> 16) | (b & 0xffff0000u); }

__device__ inline u32x4 load16(const uint16_t* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ inline void store16(uint16_t* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }

// Per-thread staging registers of one chunk's strips.
template <int SMODE>
struct StripRegs {
    static constexpr int kItems = SMODE == kStripVec ? kStripVecItems : kStripScalarItems;
    static constexpr int kWords = SMODE == kStripVec ? 32 : 4;   // item: 8 channels x 8 or 1 positions
    uint32_t d[kItems][kWords];
};

// The tile's runs, as plain values (kept in registers across the loop).
struct Runs {
    int i0, nseg, m0, qa0, d_first, d_second, d_stride, ck0, ck_mid, ck_total, start0, extent;
};

__device__ inline Runs runs_of(const TileRuns& tr, const ConvArgs& a) {
    Runs r;
    r.i0 = tr.i0; r.nseg = tr.nseg; r.m0 = tr.m0; r.qa0 = tr.qa0;
    r.d_first = tr.d_first; r.d_second = tr.d_second; r.d_stride = tr.d_stride;
    r.ck0 = tr.ck0; r.ck_mid = tr.ck_mid; r.ck_total = tr.ck_total;
    r.start0 = tr.m0 * a.row_len + tr.qa0 - tr.shift0;
    r.extent = tr.extent;
    return r;
}

// Load the strips of channels [r0, r0 + 16) into registers.
//   kStripVec:    item q = (16-byte chunk q/2 of the tile's runs, channel
//                 group q%2): 8 loads of 8 positions, one per channel
//                 (window-tensor planes are whole 16-byte vectors, so a chunk
//                 never leaves its plane);
//   kStripScalar: item q = (strip position q/2, channel group q%2), 8 loads
//                 of one window-tensor element;
//   kStripFused:  the same positions gathered from x, zero in the padding.
template <int SMODE>
__device__ inline void load_strips(StripRegs<SMODE>& R, const ConvArgs& a, const Runs& rn, int r0) {
    const uint16_t* src = static_cast<const uint16_t*>(a.src);
    if constexpr (SMODE == kStripVec) {
        const int64_t plane = (int64_t)a.ho * a.row_len;
        const int n = 2 * rn.ck_total;
#pragma unroll
        for (int k = 0; k < StripRegs<SMODE>::kItems; ++k) {
            const int q = threadIdx.x + k * kConvThreads;
            if (q < n) {
                const int c = q >> 1, g = q & 1;
                int s = 0, cs = c;
                if (c >= rn.ck0) {
                    s = 1 + (int)fast_div((uint32_t)(c - rn.ck0), a.div_ckmid);
                    if (s > rn.nseg - 1) s = rn.nseg - 1;
                    cs = c - rn.ck0 - (s - 1) * rn.ck_mid;
                }
                const int rb = r0 + 8 * g;
                const uint16_t* base = src + ((int64_t)(rn.i0 + s) * a.c + rb) * plane +
                                       (s == 0 ? rn.start0 : 0) + 8 * cs;
                if (rb + 8 <= a.c) {
#pragma unroll
                    for (int ch = 0; ch < 8; ++ch) {
                        const u32x4 v = load16(base + ch * plane);
#pragma unroll
                        for (int e = 0; e < 4; ++e) R.d[k][ch * 4 + e] = v[e];
                    }
                } else {
#pragma unroll
                    for (int ch = 0; ch < 8; ++ch) {
                        u32x4 v = {0u, 0u, 0u, 0u};
                        if (rb + ch < a.c) v = load16(base + ch * plane);
#pragma unroll
                        for (int e = 0; e < 4; ++e) R.d[k][ch * 4 + e] = v[e];
                    }
                }
            }
        }
    } else {
        const int n = 2 * rn.extent;
#pragma unroll
        for (int k = 0; k < StripRegs<SMODE>::kItems; ++k) {
            const int q = threadIdx.x + k * kConvThreads;
            if (q < n) {
                const int pos = q >> 1, g = q & 1;
                int s = 0;
                if (pos >= rn.d_second) {
                    s = 1 + (int)fast_div((uint32_t)(pos - rn.d_second), a.div_lenmid);
                    if (s > rn.nseg - 1) s = rn.nseg - 1;
                }
                const int e = pos - (s == 0 ? rn.d_first : rn.d_second + (s - 1) * rn.d_stride);
                const int in_plane = (s == 0 ? rn.m0 * a.row_len + rn.qa0 : 0) + e;
                const int rb = r0 + 8 * g;
                uint32_t v[8];
                if constexpr (SMODE == kStripScalar) {
                    const int64_t plane = (int64_t)a.ho * a.row_len;
                    const uint16_t* p = src + ((int64_t)(rn.i0 + s) * a.c + rb) * plane + in_plane;
#pragma unroll
                    for (int ch = 0; ch < 8; ++ch) v[ch] = rb + ch < a.c ? p[ch * plane] : 0u;
                } else {
                    // position (row m, column k, filter row u) of the window tensor
                    const int m = (int)fast_div((uint32_t)in_plane, a.div_row);
                    const int kq = in_plane - m * a.row_len;
                    const int kc = (int)fast_div((uint32_t)kq, a.div_fh);
                    const int u = kq - kc * a.fh;
                    const int yy = m * a.sh + u - a.ph, xx = kc - a.pw;
                    const bool inb = (unsigned)yy < (unsigned)a.h && (unsigned)xx < (unsigned)a.w_in;
                    const int64_t plane = (int64_t)a.h * a.w_in;
                    const uint16_t* p = src + ((int64_t)(rn.i0 + s) * a.c + rb) * plane +
                                        (inb ? (int64_t)yy * a.w_in + xx : 0);
#pragma unroll
                    for (int ch = 0; ch < 8; ++ch) v[ch] = (inb && rb + ch < a.c) ? p[ch * plane] : 0u;
                }
#pragma unroll
                for (int e2 = 0; e2 < 4; ++e2) R.d[k][e2] = v[2 * e2] | (v[2 * e2 + 1] << 16);
            }
        }
    }
}

// Write the loaded strips channel-innermost: S[pos][8g + ch].
template <int SMODE>
__device__ inline void store_strips(const StripRegs<SMODE>& R, uint16_t* S, const Runs& rn) {
    if constexpr (SMODE == kStripVec) {
        const int n = 2 * rn.ck_total;
#pragma unroll
        for (int k = 0; k < StripRegs<SMODE>::kItems; ++k) {
            const int q = threadIdx.x + k * kConvThreads;
            if (q < n) {
                const int c = q >> 1, g = q & 1;
                uint16_t* dst = S + (8 * c) * kRC + 8 * g;
#pragma unroll
                for (int pq = 0; pq < 8; ++pq) {
                    u32x4 o;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const uint32_t w0 = R.d[k][(2 * e) * 4 + pq / 2];
                        const uint32_t w1 = R.d[k][(2 * e + 1) * 4 + pq / 2];
                        o[e] = (pq & 1) ? hi_pair(w0, w1) : lo_pair(w0, w1);
                    }
                    store16(dst + pq * kRC, o);
                }
            }
        }
    } else {
        const int n = 2 * rn.extent;
#pragma unroll
        for (int k = 0; k < StripRegs<SMODE>::kItems; ++k) {
            const int q = threadIdx.x + k * kConvThreads;
            if (q < n) {
                const u32x4 o = {R.d[k][0], R.d[k][1], R.d[k][2], R.d[k][3]};
                store16(S + (q >> 1) * kRC + 8 * (q & 1), o);
            }
        }
    }
}

// Per-thread staging registers of one chunk's filter tile.
//   FVEC (taps T known at compile time, C*T a multiple of 8): item q =
//     (output channel q/2, channel group q%2): the 8*T consecutive filter
//     elements of 8 channels, read as T 16-byte vectors;
//   otherwise item q = (tap, output channel, channel group), 8 2-byte loads.
template <bool FVEC, int FT, int BM>
struct FilterRegs {
    static constexpr int kItems = FVEC ? (2 * BM + kConvThreads - 1) / kConvThreads : kFilterScalarItems;
    static constexpr int kWords = FVEC ? 4 * FT : 4;
    uint32_t d[kItems][kWords];
};

template <bool FVEC, int FH, int FW, int BM>
__device__ inline void load_filter(FilterRegs<FVEC, FH * FW, BM>& R, const ConvArgs& a, int j0, int r0) {
    const uint16_t* w = static_cast<const uint16_t*>(a.w);
    if constexpr (FVEC) {
        constexpr int T = FH * FW;
#pragma unroll
        for (int k = 0; k < FilterRegs<FVEC, T, BM>::kItems; ++k) {
            const int q = threadIdx.x + k * kConvThreads;
            const int j = q >> 1, g = q & 1;
            const int rb = r0 + 8 * g;
            const int nvalid_el = (a.c - rb) * T;   // elements of this group inside the filter row
            const bool ok = q < 2 * BM && j0 + j < a.k;
            const uint16_t* base = w + ((int64_t)(j0 + j) * a.c + rb) * T;
            if (ok && rb + 8 <= a.c) {
#pragma unroll
                for (int v4 = 0; v4 < T; ++v4) {
                    const u32x4 v = load16(base + 8 * v4);
#pragma unroll
                    for (int e = 0; e < 4; ++e) R.d[k][v4 * 4 + e] = v[e];
                }
            } else {
#pragma unroll
                for (int v4 = 0; v4 < T; ++v4) {
                    u32x4 v = {0u, 0u, 0u, 0u};
                    if (ok && 8 * v4 < nvalid_el) v = load16(base + 8 * v4);
#pragma unroll
                    for (int e = 0; e < 4; ++e) R.d[k][v4 * 4 + e] = v[e];
                }
            }
        }
    } else {
        const int T = a.taps;
        const int n = 2 * T * BM;
#pragma unroll
        for (int k = 0; k < FilterRegs<FVEC, FH * FW, BM>::kItems; ++k) {
            const int q = threadIdx.x + k * kConvThreads;
            const int g = q & 1, rest = q >> 1;
            const int j = rest & (BM - 1), t = rest / BM;
            const int rb = r0 + 8 * g;
            uint32_t v[8];
#pragma unroll
            for (int ch = 0; ch < 8; ++ch) v[ch] = 0u;
            if (q < n && j0 + j < a.k) {
                const int vv = (int)fast_div((uint32_t)t, a.div_fh);
                const int u = t - vv * a.fh;
                const uint16_t* p = w + ((int64_t)(j0 + j) * a.c + rb) * T + u * a.fw + vv;
#pragma unroll
                for (int ch = 0; ch < 8; ++ch) v[ch] = rb + ch < a.c ? p[ch * T] : 0u;
            }
#pragma unroll
            for (int e2 = 0; e2 < 4; ++e2) R.d[k][e2] = v[2 * e2] | (v[2 * e2 + 1] << 16);
        }
    }
}

// 16-bit element i of a register item (elements in load order)
template <int W>
__device__ inline uint32_t elem16(const uint32_t (&d)[W], int i) {
    return (i & 1) ? (d[i >> 1] >> 16) : (d[i >> 1] & 0xffffu);
}

// Write the loaded filter as F[t][j][8g + ch], t = v*Fh + u (the order of a
// window's positions); channels beyond C are zeroed here.
template <bool FVEC, int FH, int FW, int BM>
__device__ inline void store_filter(const FilterRegs<FVEC, FH * FW, BM>& R, uint16_t* F,
                                    const ConvArgs& a, int r0) {
    if constexpr (FVEC) {
        constexpr int T = FH * FW;
#pragma unroll
        for (int k = 0; k < FilterRegs<FVEC, T, BM>::kItems; ++k) {
            const int q = threadIdx.x + k * kConvThreads;
            if (q < 2 * BM) {
                const int j = q >> 1, g = q & 1;
                const int nvalid = a.c - (r0 + 8 * g);   // channels of this group inside C
#pragma unroll
                for (int v = 0; v < FW; ++v)
#pragma unroll
                    for (int u = 0; u < FH; ++u) {
                        const int t = v * FH + u, nat = u * FW + v;
                        u32x4 o;
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const uint32_t lo = 2 * e < nvalid ? elem16(R.d[k], (2 * e) * T + nat) : 0u;
                            const uint32_t hi = 2 * e + 1 < nvalid ? elem16(R.d[k], (2 * e + 1) * T + nat) : 0u;
                            o[e] = lo | (hi << 16);
                        }
                        store16(F + (t * BM + j) * kRC + 8 * g, o);
                    }
            }
        }
    } else {
        const int n = 2 * a.taps * BM;
#pragma unroll
        for (int k = 0; k < FilterRegs<FVEC, FH * FW, BM>::kItems; ++k) {
            const int q = threadIdx.x + k * kConvThreads;
            if (q < n) {
                const int g = q & 1, rest = q >> 1;
                const int j = rest & (BM - 1), t = rest / BM;
                const u32x4 o = {R.d[k][0], R.d[k][1], R.d[k][2], R.d[k][3]};
                store16(F + (t * BM + j) * kRC + 8 * g, o);
            }
        }
    }
}

__device__ inline bf16x8 frag(const uint16_t* p) { return __builtin_bit_cast(bf16x8, load16(p)); }

// MFMA over one staged chunk: for each tap, NJ filter fragments and NP window
// fragments, read from LDS one tap ahead of the matrix-core instructions that
// use them.  FT > 0 fixes the number of taps at compile time.
template <int FT, int BM, int NJ, int NP>
__device__ inline void compute_chunk(f32x16 (&acc)[NJ][NP], const uint16_t* F, const uint16_t* S,
                                     const int (&fo)[NJ], const int (&so)[NP], int taps) {
    const int T = FT > 0 ? FT : taps;
    bf16x8 a0[NJ], b0[NP], a1[NJ], b1[NP];
    auto ld = [&](bf16x8 (&av)[NJ], bf16x8 (&bv)[NP], int t) {
#pragma unroll
        for (int jb = 0; jb < NJ; ++jb) av[jb] = frag(F + t * BM * kRC + fo[jb]);
#pragma unroll
        for (int pb = 0; pb < NP; ++pb) bv[pb] = frag(S + t * kRC + so[pb]);
    };
    auto mm = [&](const bf16x8 (&av)[NJ], const bf16x8 (&bv)[NP]) {
#pragma unroll
        for (int jb = 0; jb < NJ; ++jb)
#pragma unroll
            for (int pb = 0; pb < NP; ++pb)
                acc[jb][pb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[jb], bv[pb], acc[jb][pb], 0, 0, 0);
    };
    auto pair = [&](int t) {
        ld(a1, b1, t + 1);
        mm(a0, b0);
        if (t + 2 < T) ld(a0, b0, t + 2);
        mm(a1, b1);
    };
    ld(a0, b0, 0);
    int t = 0;
    if constexpr (FT > 0) {
#pragma unroll
        for (; t + 2 <= FT; t += 2) pair(t);
    } else {
        for (; t + 2 <= T; t += 2) pair(t);
    }
    if (t < T) mm(a0, b0);
}

template <int FH, int FW, int BM, int BN, int TJ, int TP, int SMODE, bool FVEC>
__global__ __launch_bounds__(kConvThreads) void conv_bf16_kernel(ConvArgs a) {
    static_assert((BM / TJ) * (BN / TP) == kConvThreads / 64, "4 waves per workgroup");
    static_assert((BM & (BM - 1)) == 0, "BM is a power of two");
    constexpr int NJ = TJ / 32, NP = TP / 32;
    constexpr int WAVES_P = BN / TP;
    constexpr int FT = FH * FW;

    extern __shared__ __align__(16) unsigned char smem[];
    uint16_t* lds = reinterpret_cast<uint16_t*>(smem);   // stage s: S at s*stage, F after S
    const int f_off = a.strip_cap * kRC;

    const int jtile = blockIdx.x % a.num_jtiles;
    const int ptile = blockIdx.x / a.num_jtiles;
    const int j0 = jtile * BM;

    TileRuns tr;
    tr.init(ptile, BN, a);
    const Runs rn = runs_of(tr, a);

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int wj = wave / WAVES_P, wp_ = wave % WAVES_P;
    const int l32 = lane & 31, kl = lane >> 5;

    int so[NP];
    int64_t yoff[NP];
    bool pvalid[NP];
#pragma unroll
    for (int pb = 0; pb < NP; ++pb) {
        int p = tr.p0 + wp_ * TP + pb * 32 + l32;
        pvalid[pb] = p <= tr.plast;
        if (!pvalid[pb]) p = tr.p0;
        so[pb] = pixel_base(tr, a, p, &yoff[pb]) * kRC + 8 * kl;
    }
    int fo[NJ];
#pragma unroll
    for (int jb = 0; jb < NJ; ++jb) fo[jb] = (wj * TJ + jb * 32 + l32) * kRC + 8 * kl;

    f32x16 acc[NJ][NP];
#pragma unroll
    for (int jb = 0; jb < NJ; ++jb)
#pragma unroll
        for (int pb = 0; pb < NP; ++pb)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[jb][pb][v] = 0.0f;

    StripRegs<SMODE> sr;
    FilterRegs<FVEC, FT, BM> fr;
    const int nchunks = (a.c + kRC - 1) / kRC;
    load_strips<SMODE>(sr, a, rn, 0);
    load_filter<FVEC, FH, FW, BM>(fr, a, j0, 0);
    store_strips<SMODE>(sr, lds, rn);
    store_filter<FVEC, FH, FW, BM>(fr, lds + f_off, a, 0);
    // One barrier per chunk: it publishes the stage written after the MFMAs
    // of the previous chunk and tells every wave that the other stage, read
    // by those MFMAs, may be overwritten.  The next chunk's loads are issued
    // after the barrier so that the barrier does not wait for them.
    for (int ch = 0; ch < nchunks; ++ch) {
        const uint16_t* cur = lds + (ch & 1) * a.stage;
        uint16_t* nxt = lds + ((ch + 1) & 1) * a.stage;
        const bool more = ch + 1 < nchunks;
        __syncthreads();
        if (more) {
            load_strips<SMODE>(sr, a, rn, (ch + 1) * kRC);
            load_filter<FVEC, FH, FW, BM>(fr, a, j0, (ch + 1) * kRC);
        }
        compute_chunk<FT, BM, NJ, NP>(acc, cur + f_off, cur, fo, so, a.taps);
        if (more) {
            store_strips<SMODE>(sr, nxt, rn);
            store_filter<FVEC, FH, FW, BM>(fr, nxt + f_off, a, (ch + 1) * kRC);
        }
    }

    // D[row][col]: col = lane%32 (pixel), row = 8*(v/4) + 4*(lane/32) + v%4 (channel)
#pragma unroll
    for (int jb = 0; jb < NJ; ++jb)
#pragma unroll
        for (int pb = 0; pb < NP; ++pb) {
            if (!pvalid[pb]) continue;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int j = j0 + wj * TJ + jb * 32 + 8 * (v >> 2) + 4 * kl + (v & 3);
                if (j < a.k) a.y[yoff[pb] + (int64_t)j * a.howo] = acc[jb][pb][v];
            }
        }
}

template <int FH, int FW, int BM, int BN, int TJ, int TP, bool FVEC>
void launch_cfg(const ConvArgs& a, int64_t blocks, int64_t lds, int smode, hipStream_t stream) {
    auto kern = smode == kStripVec      ? conv_bf16_kernel<FH, FW, BM, BN, TJ, TP, kStripVec, FVEC>
                : smode == kStripScalar ? conv_bf16_kernel<FH, FW, BM, BN, TJ, TP, kStripScalar, FVEC>
                                        : conv_bf16_kernel<FH, FW, BM, BN, TJ, TP, kStripFused, FVEC>;
    if (lds > 64 * 1024)
        (void)hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(kConvThreads), (size_t)lds, stream, a);
}

template <int FH, int FW, bool FVEC>
void launch_tile(const ConvPlan& p, const ConvArgs& a, int64_t blocks, int smode, hipStream_t stream) {
    if (p.bm == 128) launch_cfg<FH, FW, 128, 128, 64, 64, FVEC>(a, blocks, p.lds_bytes, smode, stream);
    else if (p.bn == 128) launch_cfg<FH, FW, 64, 128, 32, 64, FVEC>(a, blocks, p.lds_bytes, smode, stream);
    else launch_cfg<FH, FW, 64, 64, 32, 32, FVEC>(a, blocks, p.lds_bytes, smode, stream);
}

// Filter sizes with a compile-time kernel (16-byte filter loads).
bool known_filter(const Geometry& g) {
    return (g.fh == 3 && g.fw == 3) || (g.fh == 3 && g.fw == 5) || (g.fh == 1 && g.fw == 1);
}

}  // namespace

// Window-tensor planes that are whole 16-byte vectors allow 16-byte strip loads.
bool bf16_strips_vec(const Geometry& g) { return ((g.ho * g.row_len) & 7) == 0; }

// Tile candidates in order of preference; the first that fits (LDS, and the
// per-thread staging registers of every strip and filter item) and gives
// every CU a workgroup is taken, else the one with the most workgroups.  When
// none fits, the bf16 problem runs on the fp32-strip kernel (inputs widened).
ConvPlan plan_conv_bf16(const Geometry& g) {
    const TileCfg large_k[] = {{128, 128}, {64, 128}, {64, 64}};
    const TileCfg small_k[] = {{64, 128}, {64, 64}};
    const TileCfg* cfgs = g.k > 64 ? large_k : small_k;
    const int ncfg = g.k > 64 ? 3 : 2;
    const bool fvec = known_filter(g) && ((g.c * g.taps) & 7) == 0;
    const bool svec = bf16_strips_vec(g);
    ConvPlan best;
    int64_t best_blocks = 0;
    for (int ci = 0; ci < ncfg; ++ci) {
        const TileCfg t = cfgs[ci];
        const int64_t cap_plain = strip_capacity(g, t.bn, 0);
        const int64_t cap_vec = strip_capacity(g, t.bn, 8);
        const int64_t cap = svec ? std::max(cap_plain, cap_vec) : cap_plain;
        if (2 * cap_plain > (int64_t)kConvThreads * kStripScalarItems) continue;
        if (svec && 2 * ((cap_vec + 7) / 8) > (int64_t)kConvThreads * kStripVecItems) continue;
        if (!fvec && 2 * g.taps * t.bm > (int64_t)kConvThreads * kFilterScalarItems) continue;
        const int64_t stage = (cap + g.taps * t.bm) * kRC;   // elements
        const int64_t lds = 2 * stage * 2;
        if (lds > kConvLdsMaxBytes) continue;
        ConvPlan p;
        p.kind = ConvPlan::kBf16Lds;
        p.bm = t.bm; p.bn = t.bn; p.rc = kRC; p.tc = (int)g.taps;
        p.strip_cap = cap; p.stage = stage; p.lds_bytes = lds;
        p.svec = svec ? 1 : 0;
        p.fvec = fvec ? 1 : 0;
        const int64_t blocks = ((g.npix + t.bn - 1) / t.bn) * ((g.k + t.bm - 1) / t.bm);
        if (blocks >= 256) return p;
        if (blocks > best_blocks) { best = p; best_blocks = blocks; }
    }
    if (best.kind != ConvPlan::kNone) return best;
    return plan_conv_f32(g);
}

ConvArgs conv_args_bf16(const Geometry& g, const ConvPlan& p, const void* src, const void* w,
                        float* y, bool fused) {
    ConvArgs a = make_conv_args(g, src, w, y, p.bm);
    a.rc = kRC;
    a.strip_cap = (int)p.strip_cap;
    a.stage = (int)p.stage;
    a.tc = p.tc;
    a.svec = (!fused && p.svec) ? 1 : 0;
    a.fvec = p.fvec;
    a.div_ckmid = make_fastdiv((uint32_t)((((g.ho - 1) * g.row_len + g.used_len) + 7) >> 3));
    return a;
}

int bf16_strip_mode(const ConvPlan& p, bool fused) {
    return fused ? kStripFused : (p.svec ? kStripVec : kStripScalar);
}

int launch_conv_bf16(const Geometry& g, bool fused, const void* src, const void* w, float* y,
                     hipStream_t stream, char* err, size_t errlen) {
    const ConvPlan p = plan_conv_bf16(g);
    if (p.kind == ConvPlan::kNone) {
        snprintf(err, errlen,
                 "conv: the window strips of one tile (row length %lld) do not fit in LDS; "
                 "this shape is not supported", (long long)g.row_len);
        return -5;
    }
    if (p.kind == ConvPlan::kF32Lds)
        return launch_conv_f32_plan(g, p, fused, src, w, y, stream, err, errlen);
    const ConvArgs a = conv_args_bf16(g, p, src, w, y, fused);
    const int64_t blocks = ((g.npix + p.bn - 1) / p.bn) * a.num_jtiles;
    if (blocks > 0x7fffffff) {
        snprintf(err, errlen, "conv: grid of %lld workgroups is too large", (long long)blocks);
        return -5;
    }
    const int smode = bf16_strip_mode(p, fused);
    if (p.fvec && g.fh == 3 && g.fw == 3) launch_tile<3, 3, true>(p, a, blocks, smode, stream);
    else if (p.fvec && g.fh == 3 && g.fw == 5) launch_tile<3, 5, true>(p, a, blocks, smode, stream);
    else if (p.fvec && g.fh == 1 && g.fw == 1) launch_tile<1, 1, true>(p, a, blocks, smode, stream);
    else launch_tile<0, 0, false>(p, a, blocks, smode, stream);
    return 0;
}

}  // namespace im2win
