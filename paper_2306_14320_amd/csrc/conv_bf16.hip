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
// Each operand is split into two planes of 8 channels (16 bytes per position)
// so that a fragment read is one 16-byte vector per lane from one plane: the
// filter planes are read contiguously, and the strip planes use a row pitch
// and image-segment bases (ClLayout) that put the windows of 16 consecutive
// pixels in 16 different bank groups when sw*Fh is odd.
//
// Neither operand has that layout in memory (the window tensor and the filter
// are channel-outer), so each chunk passes through registers:
//   - right after the barrier that opens chunk c, every thread loads its
//     items of chunk c+1: 8-byte loads of 4 strip positions for each of 8
//     channels, and 16-byte loads of one output channel's filter row for 8
//     channels and all taps; they land while the MFMAs of chunk c run;
//   - after those MFMAs the items are transposed in registers (16-bit lane
//     permutes) and written to the other of two LDS stages with 16-byte
//     stores, so one barrier per chunk suffices.
// The fused kernel gathers the strip positions from x (zero in the padding)
// with 2-byte loads, as do shapes whose window-tensor planes or filter rows
// are not whole 16-byte vectors.  Channels beyond C are zero in both
// operands.
#include "conv_common.h"

#include <cstdio>
#include <utility>

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

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ inline u32x4 load16(const uint16_t* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ inline u32x2 load8(const uint16_t* p) { return *reinterpret_cast<const u32x2*>(p); }
__device__ inline void store16(uint16_t* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }

// Per-thread staging registers of one chunk's strips.
template <int SMODE, int SVI = kStripVecItems>
struct StripRegs {
    static constexpr int kItems = SMODE == kStripVec ? SVI : kStripScalarItems;
    static constexpr int kWords = SMODE == kStripVec ? 16 : 4;   // item: 8 channels x 4 or 1 positions
    uint32_t d[kItems][kWords];
};

// The tile's runs, as plain values (kept in registers across the loop).
struct Runs {
    int i0, nseg, m0, qa0, len0, len_mid, ck0, ck_mid, ck_total, start0, strip_len;
};

__device__ inline Runs runs_of(const TileRuns& tr, const ConvArgs& a) {
    Runs r;
    r.i0 = tr.i0; r.nseg = tr.nseg; r.m0 = tr.m0; r.qa0 = tr.qa0;
    r.len0 = tr.len0; r.len_mid = tr.len_mid;
    r.ck0 = tr.ck0; r.ck_mid = tr.ck_mid; r.ck_total = tr.ck_total;
    r.start0 = tr.m0 * a.row_len + tr.qa0 - tr.shift0;
    r.strip_len = tr.strip_len;
    return r;
}

// LDS position (ClLayout) of in-plane element e of segment s.
__device__ inline int lds_pos(const ClLayout& cl, const Runs& rn, const ConvArgs& a, int s, int e) {
    const int row = (int)fast_div((uint32_t)e, a.div_row);
    return cl.seg_base(s) + (row - (s == 0 ? rn.m0 : 0)) * a.cl_pitch + (e - row * a.row_len) -
           (s == 0 ? rn.qa0 : 0);
}

// Segment and in-plane element of an item, as the loads and the stores of
// the item both need them.
struct ItemAt {
    int s, e;
};

// kStripVec: item q = (4-element group q/2 of the tile's runs, channel half
// q%2); the runs start on 4-element boundaries (shift0) and window-tensor
// planes and rows are whole groups, so a group never leaves its row.
__device__ inline ItemAt vec_item(int c, const Runs& rn, const ConvArgs& a) {
    ItemAt it;
    it.s = 0;
    int cs = c;
    if (c >= rn.ck0) {
        it.s = 1 + (int)fast_div((uint32_t)(c - rn.ck0), a.div_ckmid);
        if (it.s > rn.nseg - 1) it.s = rn.nseg - 1;
        cs = c - rn.ck0 - (it.s - 1) * rn.ck_mid;
    }
    it.e = (it.s == 0 ? rn.start0 : 0) + 4 * cs;
    return it;
}

// kStripScalar / kStripFused: item q = (run position q/2, channel half q%2),
// runs back to back in run order.
__device__ inline ItemAt scalar_item(int pos, const Runs& rn, const ConvArgs& a) {
    ItemAt it;
    it.s = 0;
    int base = 0;
    if (pos >= rn.len0) {
        it.s = 1 + (int)fast_div((uint32_t)(pos - rn.len0), a.div_lenmid);
        if (it.s > rn.nseg - 1) it.s = rn.nseg - 1;
        base = rn.len0 + (it.s - 1) * rn.len_mid;
    }
    it.e = (it.s == 0 ? rn.m0 * a.row_len + rn.qa0 : 0) + pos - base;
    return it;
}

// Load the strips of channels [r0, r0 + 16) into registers (the window
// tensor, or for the fused kernel the same positions gathered from x, zero
// in the padding).
template <int SMODE, int SVI>
__device__ inline void load_strips(StripRegs<SMODE, SVI>& R, const ConvArgs& a, const Runs& rn, int r0) {
    const uint16_t* src = static_cast<const uint16_t*>(a.src);
    if constexpr (SMODE == kStripVec) {
        // Every load is issued, with indices clamped to valid memory: a
        // thread without an item repeats item q%2 (and later stores the same
        // values to the same place), channels beyond C read channel C-1 and
        // are zeroed when stored.  Loads under no branch let the compiler
        // wait for exactly the set it is about to store.
        const int64_t plane = (int64_t)a.ho * a.row_len;
        const int n = 2 * rn.ck_total;
#pragma unroll
        for (int k = 0; k < StripRegs<SMODE, SVI>::kItems; ++k) {
            int q = threadIdx.x + k * kConvThreads;
            if (q >= n) q &= 1;
            const ItemAt it = vec_item(q >> 1, rn, a);
            const int rb = r0 + 8 * (q & 1);
            const uint16_t* base = src + (int64_t)(rn.i0 + it.s) * a.c * plane + it.e;
#pragma unroll
            for (int ch = 0; ch < 8; ++ch) {
                const int cc = rb + ch < a.c ? rb + ch : a.c - 1;
                const u32x2 v = load8(base + cc * plane);
                R.d[k][2 * ch] = v[0];
                R.d[k][2 * ch + 1] = v[1];
            }
        }
    } else {
        const int n = 2 * rn.strip_len;
#pragma unroll
        for (int k = 0; k < StripRegs<SMODE, SVI>::kItems; ++k) {
            const int q = threadIdx.x + k * kConvThreads;
            if (q < n) {
                const ItemAt it = scalar_item(q >> 1, rn, a);
                const int rb = r0 + 8 * (q & 1);
                uint32_t v[8];
                if constexpr (SMODE == kStripScalar) {
                    const int64_t plane = (int64_t)a.ho * a.row_len;
                    const uint16_t* p = src + ((int64_t)(rn.i0 + it.s) * a.c + rb) * plane + it.e;
#pragma unroll
                    for (int ch = 0; ch < 8; ++ch) v[ch] = rb + ch < a.c ? p[ch * plane] : 0u;
                } else {
                    // element (row m, column k, filter row u) of the window tensor
                    const int m = (int)fast_div((uint32_t)it.e, a.div_row);
                    const int kq = it.e - m * a.row_len;
                    const int kc = (int)fast_div((uint32_t)kq, a.div_fh);
                    const int u = kq - kc * a.fh;
                    const int yy = m * a.sh + u - a.ph, xx = kc - a.pw;
                    const bool inb = (unsigned)yy < (unsigned)a.h && (unsigned)xx < (unsigned)a.w_in;
                    const int64_t plane = (int64_t)a.h * a.w_in;
                    const uint16_t* p = src + ((int64_t)(rn.i0 + it.s) * a.c + rb) * plane +
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

// Write the loaded strips channel-innermost into the two planes:
// S + g*cl_pb*8 + pos*8 holds channels 8g .. 8g+7 of position pos.
template <int SMODE, int SVI>
__device__ inline void store_strips(const StripRegs<SMODE, SVI>& R, uint16_t* S, const Runs& rn,
                                    const ClLayout& cl, const ConvArgs& a, int r0) {
    if constexpr (SMODE == kStripVec) {
        const int n = 2 * rn.ck_total;
#pragma unroll
        for (int k = 0; k < StripRegs<SMODE, SVI>::kItems; ++k) {
            int q = threadIdx.x + k * kConvThreads;
            if (q >= n) q &= 1;
            const ItemAt it = vec_item(q >> 1, rn, a);
            uint16_t* dst = S + ((q & 1) * a.cl_pb + lds_pos(cl, rn, a, it.s, it.e)) * 8;
            uint32_t d[16];
#pragma unroll
            for (int i = 0; i < 16; ++i) d[i] = R.d[k][i];
            if (r0 + kRC > a.c) {   // last chunk: channels beyond C are zero
                const int rb = r0 + 8 * (q & 1);
#pragma unroll
                for (int ch = 0; ch < 8; ++ch)
                    if (rb + ch >= a.c) d[2 * ch] = d[2 * ch + 1] = 0u;
            }
#pragma unroll
            for (int pq = 0; pq < 4; ++pq) {
                u32x4 o;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const uint32_t w0 = d[(2 * e) * 2 + pq / 2];
                    const uint32_t w1 = d[(2 * e + 1) * 2 + pq / 2];
                    o[e] = (pq & 1) ? hi_pair(w0, w1) : lo_pair(w0, w1);
                }
                store16(dst + pq * 8, o);
            }
        }
    } else {
        const int n = 2 * rn.strip_len;
#pragma unroll
        for (int k = 0; k < StripRegs<SMODE, SVI>::kItems; ++k) {
            const int q = threadIdx.x + k * kConvThreads;
            if (q < n) {
                const ItemAt it = scalar_item(q >> 1, rn, a);
                const u32x4 o = {R.d[k][0], R.d[k][1], R.d[k][2], R.d[k][3]};
                store16(S + ((q & 1) * a.cl_pb + lds_pos(cl, rn, a, it.s, it.e)) * 8, o);
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
        // Unconditional loads with clamped indices, as for the strips: a
        // thread beyond the 2*BM items repeats one, output channels beyond K
        // read channel K-1, and 16-byte groups past the channels of the
        // filter row are clamped to its last group; all of these are zeroed
        // or duplicated when stored.
#pragma unroll
        for (int k = 0; k < FilterRegs<FVEC, T, BM>::kItems; ++k) {
            const int q = (threadIdx.x + k * kConvThreads) & (2 * BM - 1);
            const int j = q >> 1, g = q & 1;
            const int rb = r0 + 8 * g;
            const int jc = j0 + j < a.k ? j0 + j : a.k - 1;
            const int rbc = rb < a.c ? rb : (a.c - 1) & ~7;   // keeps the groups 16-byte aligned
            const int last = ((a.c - rbc) * T - 1) >> 3;   // last 16-byte group inside the row
            const uint16_t* base = w + ((int64_t)jc * a.c + rbc) * T;
#pragma unroll
            for (int v4 = 0; v4 < T; ++v4) {
                const u32x4 v = load16(base + 8 * (v4 < last ? v4 : last));
#pragma unroll
                for (int e = 0; e < 4; ++e) R.d[k][v4 * 4 + e] = v[e];
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

// Write the loaded filter into two planes, F + (g*cl_fpb + t*BM + j)*8
// holding channels 8g .. 8g+7 of tap t = v*Fh + u (the order of a window's
// positions) of output channel j; channels beyond C are zeroed here.
template <bool FVEC, int FH, int FW, int BM>
__device__ inline void store_filter(const FilterRegs<FVEC, FH * FW, BM>& R, uint16_t* F,
                                    const ConvArgs& a, int j0, int r0) {
    if constexpr (FVEC) {
        constexpr int T = FH * FW;
#pragma unroll
        for (int k = 0; k < FilterRegs<FVEC, T, BM>::kItems; ++k) {
            const int q = (threadIdx.x + k * kConvThreads) & (2 * BM - 1);
            {
                const int j = q >> 1, g = q & 1;
                // channels of this group inside C (none for output channels beyond K)
                const int nvalid = j0 + j < a.k ? a.c - (r0 + 8 * g) : 0;
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
                        store16(F + (g * a.cl_fpb + t * BM + j) * 8, o);
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
                store16(F + (g * a.cl_fpb + t * BM + j) * 8, o);
            }
        }
    }
}

__device__ inline bf16x8 frag(const uint16_t* p) { return __builtin_bit_cast(bf16x8, load16(p)); }

// Repack K x C x Fh x Fw into the blocks of packed_piece().  Workgroup
// (row group jg, chunk ch) copies the 16*T filter elements of chunk ch of
// output channels kPackRows*jg .. +kPackRows-1 (one contiguous run per output
// channel) to LDS, then writes its 2*T*kPackRows pieces: for each (half g,
// tap t) the kPackRows pieces of consecutive output channels are
// consecutive in the packed tensor.
__global__ __launch_bounds__(256) void pack_filter_bf16_kernel(const uint16_t* __restrict__ w,
                                                               uint16_t* __restrict__ wp, int c, int fh,
                                                               int fw, int bm, int nchunks) {
    extern __shared__ __align__(16) unsigned char smem[];
    uint16_t* L = reinterpret_cast<uint16_t*>(smem);   // [kPackRows][16*T]
    const int T = fh * fw, run = kBf16ChunkChannels * T;
    const int ch = blockIdx.x % nchunks, jg = blockIdx.x / nchunks;
    const int j0 = jg * kPackRows;
    // 2-byte elements (runs start at even element offsets only when T is even)
#pragma unroll
    for (int r = 0; r < kPackRows; ++r) {
        const uint16_t* src = w + ((int64_t)(j0 + r) * c + kBf16ChunkChannels * ch) * T;
        for (int q = threadIdx.x; q < run; q += 256) L[r * run + q] = src[q];
    }
    __syncthreads();
    for (int pc = threadIdx.x; pc < 2 * T * kPackRows; pc += 256) {
        const int jj = pc % kPackRows, gt = pc / kPackRows;   // gt = g*T + t
        const int g = gt >= T ? 1 : 0, t = gt - g * T;
        const int v = t / fh, u = t - v * fh, nat = u * fw + v;
        const uint16_t* s = L + jj * run + 8 * g * T + nat;
        u32x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = uint32_t(s[(2 * e) * T]) | (uint32_t(s[(2 * e + 1) * T]) << 16);
        store16(wp + packed_index(j0 + jj, ch, g, t, T, bm, nchunks) * 8, o);
    }
}

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
        for (int jb = 0; jb < NJ; ++jb) av[jb] = frag(F + t * BM * 8 + fo[jb]);
#pragma unroll
        for (int pb = 0; pb < NP; ++pb) bv[pb] = frag(S + t * 8 + so[pb]);
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

template <int FH, int FW, int BM, int BN, int TJ, int TP, int SMODE, bool FVEC, int SVI>
__global__ __launch_bounds__(kConvThreads) void conv_bf16_kernel(ConvArgs a) {
    static_assert((BM / TJ) * (BN / TP) == kConvThreads / 64, "4 waves per workgroup");
    static_assert((BM & (BM - 1)) == 0, "BM is a power of two");
    constexpr int NJ = TJ / 32, NP = TP / 32;
    constexpr int WAVES_P = BN / TP;
    constexpr int FT = FH * FW;

    extern __shared__ __align__(16) unsigned char smem[];
    uint16_t* lds = reinterpret_cast<uint16_t*>(smem);   // stage s: strip planes, then filter planes
    const int f_off = 2 * a.cl_pb * 8;

    const int jtile = blockIdx.x % a.num_jtiles;
    const int ptile = blockIdx.x / a.num_jtiles;
    const int j0 = jtile * BM;

    TileRuns tr;
    tr.init(ptile, BN, a);
    const Runs rn = runs_of(tr, a);
    const ClLayout cl = cl_layout(tr, a);

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
        so[pb] = (kl * a.cl_pb + cl_pixel_base(cl, tr, a, p, &yoff[pb])) * 8;
    }
    int fo[NJ];
#pragma unroll
    for (int jb = 0; jb < NJ; ++jb) fo[jb] = (kl * a.cl_fpb + wj * TJ + jb * 32 + l32) * 8;

    f32x16 acc[NJ][NP];
#pragma unroll
    for (int jb = 0; jb < NJ; ++jb)
#pragma unroll
        for (int pb = 0; pb < NP; ++pb)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[jb][pb][v] = 0.0f;

    // Two register sets: chunk k is staged through set k % 2.  Its loads are
    // issued right after the barrier that opens chunk k - 2, so they have two
    // chunks of MFMA work to land; after the MFMAs of chunk k - 1 the set is
    // transposed into the LDS stage of chunk k.  One barrier per chunk
    // publishes that stage and frees the other one; it waits for LDS
    // operations only, not for the loads still in flight.
    StripRegs<SMODE, SVI> sr0, sr1;
    FilterRegs<FVEC, FT, BM> fr0, fr1;
    const int nchunks = (a.c + kRC - 1) / kRC;
    load_strips<SMODE, SVI>(sr0, a, rn, 0);
    load_filter<FVEC, FH, FW, BM>(fr0, a, j0, 0);
    store_strips<SMODE, SVI>(sr0, lds, rn, cl, a, 0);
    store_filter<FVEC, FH, FW, BM>(fr0, lds + f_off, a, j0, 0);
    if (nchunks > 1) {
        load_strips<SMODE, SVI>(sr1, a, rn, kRC);
        load_filter<FVEC, FH, FW, BM>(fr1, a, j0, kRC);
    }
    auto step = [&](int ch, StripRegs<SMODE, SVI>& s_ld, FilterRegs<FVEC, FT, BM>& f_ld,
                    StripRegs<SMODE, SVI>& s_st, FilterRegs<FVEC, FT, BM>& f_st) {
        const uint16_t* cur = lds + (ch & 1) * a.stage;
        uint16_t* nxt = lds + ((ch + 1) & 1) * a.stage;
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
        if (ch + 2 < nchunks) {
            load_strips<SMODE, SVI>(s_ld, a, rn, (ch + 2) * kRC);
            load_filter<FVEC, FH, FW, BM>(f_ld, a, j0, (ch + 2) * kRC);
        }
        compute_chunk<FT, BM, NJ, NP>(acc, cur + f_off, cur, fo, so, a.taps);
        if (ch + 1 < nchunks) {
            store_strips<SMODE, SVI>(s_st, nxt, rn, cl, a, (ch + 1) * kRC);
            store_filter<FVEC, FH, FW, BM>(f_st, nxt + f_off, a, j0, (ch + 1) * kRC);
        }
    };
    int ch = 0;
    for (; ch + 2 <= nchunks; ch += 2) {
        step(ch, sr0, fr0, sr1, fr1);
        step(ch + 1, sr1, fr1, sr0, fr0);
    }
    if (ch < nchunks) step(ch, sr0, fr0, sr1, fr1);

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

// The common case, as one branch-free loop: strips in 4-element groups and
// filter rows in 16-byte vectors (both operands whole vectors), C a multiple
// of the 16-channel chunk and K of the tile's channels.  The item addresses
// are the same for every chunk but for the channel offset, so they are
// computed once; the stores of chunk c+1 (transposes + 16-byte LDS writes,
// one filter tap and one strip position per step) are interleaved with the
// MFMAs of chunk c, which a single wave per SIMD cannot otherwise overlap.
// Chunks past the last are loaded again from the last one and written to the
// stage no MFMA reads any more, so no step needs a branch.
// Per-thread staging registers of one chunk (unfused fast kernel): strips
// and packed filter pieces.
template <int SVI, int FI>
struct FastStage {
    uint32_t sd[SVI][16];          // strips: 8 channels x 4 positions per item
    u32x4 fd[FI];                  // packed filter pieces threadIdx.x + NT*i
};

// Unfused kernel for the common case: whole 16-channel chunks, whole tiles of
// output channels, window-tensor planes and rows of whole 4-element groups.
// The filter comes packed (packed_piece): a thread's pieces go to LDS
// unchanged.  Strips and filter pieces pass through registers two chunks
// ahead, so every global load is one the compiler waits for precisely, and
// the chunk barrier only waits for the LDS stores.
// NT threads per workgroup: 256 (4 waves), or 512 (8 waves, two per SIMD
// when one workgroup fills a CU).
template <int FH, int FW, int BM, int BN, int TJ, int TP, int SVI, int NT>
__global__ __launch_bounds__(NT) void conv_bf16_fast_kernel(ConvArgs a) {
    static_assert((BM / TJ) * (BN / TP) == NT / 64, "one wave per TJ x TP block");
    constexpr int NJ = TJ / 32, NP = TP / 32;
    constexpr int WAVES_P = BN / TP;
    constexpr int T = FH * FW;
    constexpr int kPlane = T * BM, kPieces = 2 * kPlane;
    constexpr int FI = (kPieces + NT - 1) / NT;   // filter pieces per thread
    static_assert(FI <= T, "one filter piece stored per tap");
    using St = FastStage<SVI, FI>;

    extern __shared__ __align__(16) unsigned char smem[];
    uint16_t* lds = reinterpret_cast<uint16_t*>(smem);
    const int f_off = 2 * a.cl_pb * 8;

    const int jtile = blockIdx.x % a.num_jtiles;
    const int ptile = blockIdx.x / a.num_jtiles;
    const int j0 = jtile * BM;

    TileRuns tr;
    tr.init(ptile, BN, a);
    const Runs rn = runs_of(tr, a);
    const ClLayout cl = cl_layout(tr, a);

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
        so[pb] = (kl * a.cl_pb + cl_pixel_base(cl, tr, a, p, &yoff[pb])) * 8;
    }
    int fo[NJ];
#pragma unroll
    for (int jb = 0; jb < NJ; ++jb) fo[jb] = (kl * a.cl_fpb + wj * TJ + jb * 32 + l32) * 8;

    // per-item sources (channel 0 of the chunk) and LDS destinations
    const uint16_t* src = static_cast<const uint16_t*>(a.src);
    const int plane = a.ho * a.row_len;
    const uint16_t* sp[SVI];
    int sdst[SVI];
    const int nitems = 2 * rn.ck_total;
#pragma unroll
    for (int k = 0; k < SVI; ++k) {
        int q = threadIdx.x + k * NT;
        if (q >= nitems) q &= 1;          // repeat an item: same values, same place
        const ItemAt it = vec_item(q >> 1, rn, a);
        sp[k] = src + ((int64_t)(rn.i0 + it.s) * a.c + 8 * (q & 1)) * plane + it.e;
        sdst[k] = ((q & 1) * a.cl_pb + lds_pos(cl, rn, a, it.s, it.e)) * 8;
    }
    const int nchunks = a.c / kRC;
    // packed filter blocks of this tile of output channels; this thread's
    // pieces P = threadIdx.x + NT*i and their LDS positions (the last piece
    // again, never stored, where P runs past the block)
    const uint16_t* fblk = static_cast<const uint16_t*>(a.w) + (int64_t)jtile * nchunks * (16 * T * BM);
    int fpc[FI], fdst[FI];
#pragma unroll
    for (int i = 0; i < FI; ++i) {
        const int P = threadIdx.x + NT * i;
        const int Pc = P < kPieces ? P : kPieces - 1;
        const int g = Pc >= kPlane ? 1 : 0;
        fpc[i] = Pc * 8;
        fdst[i] = f_off + (g * a.cl_fpb + Pc - g * kPlane) * 8;
    }

    St st0, st1;
    auto load = [&](St& r, int ch) {
        const int chc = ch < nchunks ? ch : nchunks - 1;
        const uint16_t* fb = fblk + (int64_t)chc * (16 * T * BM);
#pragma unroll
        for (int i = 0; i < FI; ++i) r.fd[i] = load16(fb + fpc[i]);
        const int r0 = chc * kRC;
#pragma unroll
        for (int k = 0; k < SVI; ++k) {
            const uint16_t* p = sp[k] + (int64_t)r0 * plane;
#pragma unroll
            for (int c8 = 0; c8 < 8; ++c8) {
                const u32x2 v = load8(p + c8 * plane);
                r.sd[k][2 * c8] = v[0];
                r.sd[k][2 * c8 + 1] = v[1];
            }
        }
    };
    // part t of the stores of one stage: filter piece t (t < FI), and strip
    // position t (t < 4) of every item (16-bit transpose, one 16-byte store)
    auto part = [&](const St& r, uint16_t* stg, int t) {
        const int ti = t < FI ? t : 0;   // (indices stay inside the arrays when t >= FI)
        if (t < FI && threadIdx.x + NT * t < kPieces) store16(stg + fdst[ti], r.fd[ti]);
        if (t >= 4) return;
#pragma unroll
        for (int k = 0; k < SVI; ++k) {
            u32x4 o;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const uint32_t w0 = r.sd[k][(2 * e) * 2 + t / 2];
                const uint32_t w1 = r.sd[k][(2 * e + 1) * 2 + t / 2];
                o[e] = (t & 1) ? hi_pair(w0, w1) : lo_pair(w0, w1);
            }
            store16(stg + sdst[k] + t * 8, o);
        }
    };

    f32x16 acc[NJ][NP];
#pragma unroll
    for (int jb = 0; jb < NJ; ++jb)
#pragma unroll
        for (int pb = 0; pb < NP; ++pb)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[jb][pb][v] = 0.0f;

    // chunk 0 into stage 0; chunk 1 in flight
    load(st0, 0);
#pragma unroll
    for (int t = 0; t < (T > 4 ? T : 4); ++t) part(st0, lds, t);
    load(st1, 1);

    auto step = [&](int ch, St& r_ld, St& r_st) {
        const uint16_t* cur = lds + (ch & 1) * a.stage;
        uint16_t* nxt = lds + ((ch + 1) & 1) * a.stage;
        // chunk ch complete in LDS (this wave's stores, then everyone's), and
        // every wave done with chunk ch-1, whose stage is refilled below
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
        load(r_ld, ch + 2);
        __builtin_amdgcn_sched_barrier(0);   // keep the copies at the head of the step
        const uint16_t* F = cur + f_off;
        auto ld = [&](bf16x8 (&av)[NJ], bf16x8 (&bv)[NP], int t) {
#pragma unroll
            for (int jb = 0; jb < NJ; ++jb) av[jb] = frag(F + t * BM * 8 + fo[jb]);
#pragma unroll
            for (int pb = 0; pb < NP; ++pb) bv[pb] = frag(cur + t * 8 + so[pb]);
        };
        auto mm = [&](const bf16x8 (&av)[NJ], const bf16x8 (&bv)[NP]) {
#pragma unroll
            for (int jb = 0; jb < NJ; ++jb)
#pragma unroll
                for (int pb = 0; pb < NP; ++pb)
                    acc[jb][pb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[jb], bv[pb], acc[jb][pb], 0, 0, 0);
        };
        // operands read two taps ahead of the matrix-core instructions
        bf16x8 av[3][NJ], bv[3][NP];
        ld(av[0], bv[0], 0);
        if (1 < T) ld(av[1], bv[1], 1);
#pragma unroll
        for (int t = 0; t < T; ++t) {
            if (t + 2 < T) ld(av[(t + 2) % 3], bv[(t + 2) % 3], t + 2);
            mm(av[t % 3], bv[t % 3]);
            part(r_st, nxt, t);
        }
#pragma unroll
        for (int t2 = T; t2 < 4; ++t2) part(r_st, nxt, t2);   // strip positions when T < 4
    };
    int ch = 0;
    for (; ch + 2 <= nchunks; ch += 2) {
        step(ch, st0, st1);
        step(ch + 1, st1, st0);
    }
    if (ch < nchunks) step(ch, st0, st1);

    // D[row][col]: col = lane%32 (pixel), row = 8*(v/4) + 4*(lane/32) + v%4 (channel)
#pragma unroll
    for (int jb = 0; jb < NJ; ++jb)
#pragma unroll
        for (int pb = 0; pb < NP; ++pb) {
            if (!pvalid[pb]) continue;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int j = j0 + wj * TJ + jb * 32 + 8 * (v >> 2) + 4 * kl + (v & 3);
                a.y[yoff[pb] + (int64_t)j * a.howo] = acc[jb][pb][v];
            }
        }
}

// Fused kernel for the same common case, and x rows of an even number of
// elements: the strips are built on chip from the input rows the tile uses.
// An item is a pair of neighbouring input elements of one row for the 8
// channels of one half.  Each thread loads its item (eight 4-byte loads, one
// per channel) and its packed filter pieces two chunks ahead, in registers;
// while the MFMAs of chunk c run it transposes the item of chunk c+1 to two
// 8-channel positions and writes them to every strip position that holds
// them, one per window row m with filter row u = y + ph - m*sh, and stores
// its filter pieces.  The destinations do not change between chunks, so they
// are computed once; the ones outside the tile's runs go to the lane's own
// spare slot at the end of the strip plane.  Every global load is one the
// compiler waits for, so the chunk barrier only waits for the LDS stores.
// Padding positions are zeroed once.
template <int FH>
struct FusedMap {
    int dst[2][FH];   // element offsets in a stage of the two positions, per window-row slot
};

// NT threads per workgroup, as for the fast kernel.
template <int FH, int FW, int BM, int BN, int TJ, int TP, int IPT, int NT>
__global__ __launch_bounds__(NT) void conv_bf16_fused_kernel(ConvArgs a) {
    static_assert((BM / TJ) * (BN / TP) == NT / 64, "one wave per TJ x TP block");
    static_assert(IPT >= 1 && IPT <= kBf16FusedItems, "raw items per thread");
    constexpr int NJ = TJ / 32, NP = TP / 32;
    constexpr int WAVES_P = BN / TP;
    constexpr int T = FH * FW;

    extern __shared__ __align__(16) unsigned char smem[];
    uint16_t* lds = reinterpret_cast<uint16_t*>(smem);
    const int f_off = 2 * a.cl_pb * 8;

    const int jtile = blockIdx.x % a.num_jtiles;
    const int ptile = blockIdx.x / a.num_jtiles;
    const int j0 = jtile * BM;

    TileRuns tr;
    tr.init(ptile, BN, a);
    const ClLayout cl = cl_layout(tr, a);
    const RawRows rr = raw_rows(tr, a);

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
        so[pb] = (kl * a.cl_pb + cl_pixel_base(cl, tr, a, p, &yoff[pb])) * 8;
    }
    int fo[NJ];
#pragma unroll
    for (int jb = 0; jb < NJ; ++jb) fo[jb] = (kl * a.cl_fpb + wj * TJ + jb * 32 + l32) * 8;

    const uint16_t* xsrc = static_cast<const uint16_t*>(a.src);
    const int64_t xplane = (int64_t)a.h * a.w_in;
    const int nitems = rr.rtot * a.w_in;   // (rtot*W/2 pairs) x 2 halves

    // item q: half g = q & 1, element pair e0 = 2*(q >> 1) of the raw rows
    // -> raw row r, column xx (even), segment s, input row yy
    auto item_at = [&](int q, int* s, int* yy, int* xx) {
        const int e0 = 2 * (q >> 1);
        const int r = (int)fast_div((uint32_t)e0, a.div_w);
        *xx = e0 - r * a.w_in;
        *s = r < rr.r0 ? 0 : 1 + (int)fast_div((uint32_t)(r - rr.r0), a.div_rmid);
        if (*s > tr.nseg - 1) *s = tr.nseg - 1;
        *yy = *s == 0 ? rr.ylo0 + r : a.ylo_mid + (r - rr.r0 - (*s - 1) * a.rmid);
    };
    // item sources: channel 0 of the thread's items (items past nitems load
    // item q & 1 instead, a valid address, and are never expanded)
    int64_t xbase[IPT];
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
        int q = threadIdx.x + j * NT;
        if (q >= nitems) q &= 1;
        int sg, yy, xx;
        item_at(q, &sg, &yy, &xx);
        xbase[j] = ((int64_t)(tr.i0 + sg) * a.c + 8 * (q & 1)) * xplane + (int64_t)yy * a.w_in + xx;
    }
    // expansion map of this thread's items
    FusedMap<FH> mp[IPT];
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
        const int q = threadIdx.x + j * NT;
        const int g = q & 1;
        const int spare = (g * a.cl_pb + a.cl_pb - kBf16Spare + lane) * 8;
#pragma unroll
        for (int i = 0; i < FH; ++i) mp[j].dst[0][i] = mp[j].dst[1][i] = spare;
        if (q < nitems) {
            int sg, yy, xx;
            item_at(q, &sg, &yy, &xx);
            const int m_st = sg == 0 ? tr.m0 : 0, q_st = sg == 0 ? tr.qa0 : 0;
            const int len = sg == 0 ? tr.len0 : (sg == tr.nseg - 1 ? tr.len_last : tr.len_mid);
            const int m_end = sg == tr.nseg - 1 ? tr.m1 : a.ho - 1;
            const int t0 = yy + a.ph - a.fh + 1;
            int m_lo = t0 <= 0 ? 0 : (int)fast_div((uint32_t)(t0 + a.sh - 1), a.div_sh);
            if (m_lo < m_st) m_lo = m_st;
            int m_hi = (int)fast_div((uint32_t)(yy + a.ph), a.div_sh);
            if (m_hi > m_end) m_hi = m_end;
#pragma unroll
            for (int i = 0; i < FH; ++i) {
                const int m = m_lo + i;
                if (m > m_hi) continue;
                const int u = yy + a.ph - m * a.sh;
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int e_in = m * a.row_len + (xx + h + a.pw) * a.fh + u;
                    const int rel = e_in - (m_st * a.row_len + q_st);
                    // (columns past a trimmed row's end are skipped)
                    if (xx + h < a.w_in && (unsigned)rel < (unsigned)len && xx + h + a.pw < a.wp)
                        mp[j].dst[h][i] = (g * a.cl_pb + cl_pos(cl, tr, a, sg, e_in)) * 8;
                }
            }
        }
    }
    const int nchunks = a.c / kRC;
    // packed filter blocks of this tile of output channels, and this thread's
    // pieces P = threadIdx.x + NT*i (the last piece again, never stored,
    // where P runs past the block)
    constexpr int kPlane = T * BM, kPieces = 2 * kPlane;
    constexpr int FI = (kPieces + NT - 1) / NT;
    static_assert(FI <= T && FH <= T, "one filter piece and one window-row slot stored per tap");
    const uint16_t* fblk = static_cast<const uint16_t*>(a.w) + (int64_t)jtile * nchunks * (16 * T * BM);
    int fpc[FI], fdst[FI];
#pragma unroll
    for (int i = 0; i < FI; ++i) {
        const int P = threadIdx.x + NT * i;
        const int Pc = P < kPieces ? P : kPieces - 1;
        const int g = Pc >= kPlane ? 1 : 0;
        fpc[i] = Pc * 8;
        fdst[i] = f_off + (g * a.cl_fpb + Pc - g * kPlane) * 8;
    }
    struct Stage {
        uint32_t xd[IPT][8];   // item: 2 elements x 8 channels
        u32x4 fd[FI];
    };
    auto load = [&](Stage& r, int ch) {
        const int chc = ch < nchunks ? ch : nchunks - 1;
        const uint16_t* fb = fblk + (int64_t)chc * (16 * T * BM);
#pragma unroll
        for (int i = 0; i < FI; ++i) r.fd[i] = load16(fb + fpc[i]);
        const int64_t off = (int64_t)chc * kRC * xplane;
#pragma unroll
        for (int j = 0; j < IPT; ++j)
#pragma unroll
            for (int c8 = 0; c8 < 8; ++c8)
                r.xd[j][c8] = *reinterpret_cast<const uint32_t*>(xsrc + xbase[j] + off + c8 * xplane);
    };
    // part t of the stores of one stage: filter piece t (t < FI), and window
    // row slot t (t < FH) of both positions of every item
    auto part = [&](const Stage& r, uint16_t* stg, int t) {
        const int ti = t < FI ? t : 0;
        if (t < FI && threadIdx.x + NT * t < kPieces) store16(stg + fdst[ti], r.fd[ti]);
        if (t >= FH) return;
        const int tu = t < FH ? t : 0;
#pragma unroll
        for (int j = 0; j < IPT; ++j) {
            if (threadIdx.x + j * NT < nitems) {
                u32x4 o0, o1;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    o0[e] = lo_pair(r.xd[j][2 * e], r.xd[j][2 * e + 1]);
                    o1[e] = hi_pair(r.xd[j][2 * e], r.xd[j][2 * e + 1]);
                }
                store16(stg + mp[j].dst[0][tu], o0);
                store16(stg + mp[j].dst[1][tu], o1);
            }
        }
    };

    f32x16 acc[NJ][NP];
#pragma unroll
    for (int jb = 0; jb < NJ; ++jb)
#pragma unroll
        for (int pb = 0; pb < NP; ++pb)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[jb][pb][v] = 0.0f;

    // strip planes of both stages start at zero (the padding stays zero)
    {
        const u32x4 z = {0u, 0u, 0u, 0u};
        for (int st = 0; st < 2; ++st)
            for (int e = threadIdx.x; e < 2 * a.cl_pb; e += NT) store16(lds + st * a.stage + e * 8, z);
    }
    Stage st0, st1;
    load(st0, 0);
    load(st1, 1);
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");   // zeros before strips
#pragma unroll
    for (int t = 0; t < T; ++t) part(st0, lds, t);

    auto step = [&](int ch, Stage& r_ld, Stage& r_st) {
        const uint16_t* cur = lds + (ch & 1) * a.stage;
        uint16_t* nxt = lds + ((ch + 1) & 1) * a.stage;
        // chunk ch complete in LDS (this wave's stores, then everyone's), and
        // every wave done with chunk ch-1, whose stage is refilled below
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
        load(r_ld, ch + 2);
        __builtin_amdgcn_sched_barrier(0);
        const uint16_t* F = cur + f_off;
        auto ld = [&](bf16x8 (&av)[NJ], bf16x8 (&bv)[NP], int t) {
#pragma unroll
            for (int jb = 0; jb < NJ; ++jb) av[jb] = frag(F + t * BM * 8 + fo[jb]);
#pragma unroll
            for (int pb = 0; pb < NP; ++pb) bv[pb] = frag(cur + t * 8 + so[pb]);
        };
        auto mm = [&](const bf16x8 (&av)[NJ], const bf16x8 (&bv)[NP]) {
#pragma unroll
            for (int jb = 0; jb < NJ; ++jb)
#pragma unroll
                for (int pb = 0; pb < NP; ++pb)
                    acc[jb][pb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[jb], bv[pb], acc[jb][pb], 0, 0, 0);
        };
        bf16x8 av[3][NJ], bv[3][NP];
        ld(av[0], bv[0], 0);
        if (1 < T) ld(av[1], bv[1], 1);
#pragma unroll
        for (int t = 0; t < T; ++t) {
            if (t + 2 < T) ld(av[(t + 2) % 3], bv[(t + 2) % 3], t + 2);
            mm(av[t % 3], bv[t % 3]);
            if (ch + 1 < nchunks) part(r_st, nxt, t);
        }
    };
    int ch = 0;
    for (; ch + 2 <= nchunks; ch += 2) {
        step(ch, st0, st1);
        step(ch + 1, st1, st0);
    }
    if (ch < nchunks) step(ch, st0, st1);

#pragma unroll
    for (int jb = 0; jb < NJ; ++jb)
#pragma unroll
        for (int pb = 0; pb < NP; ++pb) {
            if (!pvalid[pb]) continue;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int j = j0 + wj * TJ + jb * 32 + 8 * (v >> 2) + 4 * kl + (v & 3);
                a.y[yoff[pb] + (int64_t)j * a.howo] = acc[jb][pb][v];
            }
        }
}

template <int FH, int FW, int BM, int BN, int TJ, int TP, bool FVEC>
void launch_cfg(const ConvArgs& a, int64_t blocks, int64_t lds, int smode, int svi, hipStream_t stream) {
    auto kern = smode == kStripVec      ? (svi == 1 ? conv_bf16_kernel<FH, FW, BM, BN, TJ, TP, kStripVec, FVEC, 1>
                                                    : conv_bf16_kernel<FH, FW, BM, BN, TJ, TP, kStripVec, FVEC, 2>)
                : smode == kStripScalar ? conv_bf16_kernel<FH, FW, BM, BN, TJ, TP, kStripScalar, FVEC, 1>
                                        : conv_bf16_kernel<FH, FW, BM, BN, TJ, TP, kStripFused, FVEC, 1>;
    if (lds > 64 * 1024)
        (void)hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(kConvThreads), (size_t)lds, stream, a);
}

template <int FH, int FW, int BM, int BN, int TJ, int TP, int NT = kConvThreads>
void launch_fast_cfg(const ConvArgs& a, int64_t blocks, int64_t lds, int svi, hipStream_t stream) {
    auto kern = svi == 1 ? conv_bf16_fast_kernel<FH, FW, BM, BN, TJ, TP, 1, NT>
                         : conv_bf16_fast_kernel<FH, FW, BM, BN, TJ, TP, 2, NT>;
    if (lds > 64 * 1024)
        (void)hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(NT), (size_t)lds, stream, a);
}

template <int FH, int FW, int BM, int BN, int TJ, int TP, int NT = kConvThreads>
void launch_fused_cfg(const ConvArgs& a, int64_t blocks, int64_t lds, int ipt, hipStream_t stream) {
    auto kern = ipt == 1 ? conv_bf16_fused_kernel<FH, FW, BM, BN, TJ, TP, 1, NT>
                         : conv_bf16_fused_kernel<FH, FW, BM, BN, TJ, TP, 2, NT>;
    if (lds > 64 * 1024)
        (void)hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(NT), (size_t)lds, stream, a);
}

template <int FH, int FW, bool FVEC>
void launch_tile(const ConvPlan& p, const ConvArgs& a, int64_t blocks, int smode, hipStream_t stream) {
    const int svi = p.strip_items > kConvThreads ? 2 : 1;
    if constexpr (FVEC && FH <= 3) {
        if (smode == kStripFused && p.fused_fast) {
            const int ipt = p.fused_ipt;
            // (8 waves of 64 x 64; the plan holds at most 512 raw items then)
            if (p.bn == 256) launch_fused_cfg<FH, FW, 128, 256, 64, 64, 512>(a, blocks, p.lds_bytes, 1, stream);
            else if (p.bm == 128) launch_fused_cfg<FH, FW, 128, 128, 64, 64>(a, blocks, p.lds_bytes, ipt, stream);
            else if (p.bn == 128) launch_fused_cfg<FH, FW, 64, 128, 32, 64>(a, blocks, p.lds_bytes, ipt, stream);
            else launch_fused_cfg<FH, FW, 64, 64, 32, 32>(a, blocks, p.lds_bytes, ipt, stream);
            return;
        }
    }
    if constexpr (FVEC) {
        if (smode == kStripVec && p.fast) {
            // the 128 x 256 tile runs one workgroup per CU: 8 waves of 64 x 64,
            // two per SIMD
            if (p.bn == 256)
                launch_fast_cfg<FH, FW, 128, 256, 64, 64, 512>(a, blocks, p.lds_bytes, p.strip_items > 512 ? 2 : 1, stream);
            else if (p.bm == 128) launch_fast_cfg<FH, FW, 128, 128, 64, 64>(a, blocks, p.lds_bytes, svi, stream);
            else if (p.bn == 128) launch_fast_cfg<FH, FW, 64, 128, 32, 64>(a, blocks, p.lds_bytes, svi, stream);
            else launch_fast_cfg<FH, FW, 64, 64, 32, 32>(a, blocks, p.lds_bytes, svi, stream);
            return;
        }
    }
    if (p.bm == 128) launch_cfg<FH, FW, 128, 128, 64, 64, FVEC>(a, blocks, p.lds_bytes, smode, svi, stream);
    else if (p.bn == 128) launch_cfg<FH, FW, 64, 128, 32, 64, FVEC>(a, blocks, p.lds_bytes, smode, svi, stream);
    else launch_cfg<FH, FW, 64, 64, 32, 32, FVEC>(a, blocks, p.lds_bytes, smode, svi, stream);
}

// Filter sizes with a compile-time kernel (16-byte filter loads).
bool known_filter(const Geometry& g) {
    return (g.fh == 3 && g.fw == 3) || (g.fh == 3 && g.fw == 5) || (g.fh == 1 && g.fw == 1);
}

}  // namespace

// Strips are loaded in groups of 4 elements (8 bytes) when window-tensor
// planes and rows are whole groups.
bool bf16_strips_vec(const Geometry& g) { return ((g.ho * g.row_len) & 3) == 0 && (g.row_len & 3) == 0; }

// LDS row pitch of the channel-inner strips: congruent to sw*Fh*Wo mod 16.
int64_t bf16_cl_pitch(const Geometry& g) {
    return g.row_len + mod16((int)((g.sw * g.fh * g.wo - g.row_len) % 16));
}

// Tile candidates in order of preference; the first that fits (LDS, and the
// per-thread staging registers of every strip and filter item) and gives
// every CU a workgroup is taken, else the one with the most workgroups.  When
// none fits, the bf16 problem runs on the fp32-strip kernel (inputs widened).
ConvPlan plan_conv_bf16(const Geometry& g, bool fused) {
    const TileCfg large_k[] = {{128, 128}, {64, 128}, {64, 64}};
    const TileCfg small_k[] = {{64, 128}, {64, 64}};
    const TileCfg* cfgs = g.k > 64 ? large_k : small_k;
    const int ncfg = g.k > 64 ? 3 : 2;
    const bool fvec = known_filter(g) && ((g.c * g.taps) & 7) == 0;
    const bool svec = bf16_strips_vec(g);
    const int64_t pitch = bf16_cl_pitch(g);
    ConvPlan best;
    int64_t best_blocks = 0;
    for (int ci = 0; ci < ncfg; ++ci) {
        const TileCfg t = cfgs[ci];
        const int64_t run_plain = strip_capacity(g, t.bn, 0);
        const int64_t run_vec = strip_capacity(g, t.bn, 4);
        if (2 * run_plain > (int64_t)kConvThreads * kStripScalarItems) continue;
        const int64_t vec_items = 2 * ((run_vec + 3) / 4);   // 4-element groups x 2 halves
        if (svec && vec_items > (int64_t)kConvThreads * kStripVecItems) continue;
        if (!fvec && 2 * g.taps * t.bm > (int64_t)kConvThreads * kFilterScalarItems) continue;
        const int64_t ext = cl_extent_bound(g, t.bn, pitch) + kBf16Spare;
        const int64_t pb = ext + mod16((int)((2 - ext) % 16));       // = 2 mod 16
        const int64_t fpb = g.taps * t.bm + 8;                        // = 8 mod 16
        const int64_t stage = 16 * (pb + fpb);                       // elements
        const int64_t lds = 2 * stage * 2;
        if (lds > kConvLdsMaxBytes || stage > (int64_t(1) << 30)) continue;
        // fused kernel from raw row items: whole 16-channel chunks, whole
        // tiles of output channels, even rows, filters of up to 3 rows,
        // and the items of every tile in the per-thread registers and LDS
        const int64_t raw_items = raw_rows_bound(g, t.bn) * g.w;   // per chunk and tile
        const bool fused_fast = fvec && g.c % kRC == 0 && g.k % t.bm == 0 && g.w % 2 == 0 && g.fh <= 3 &&
                                raw_items <= (int64_t)kConvThreads * kBf16FusedItems;
        ConvPlan p;
        p.kind = ConvPlan::kBf16Lds;
        p.bm = t.bm; p.bn = t.bn; p.rc = kRC; p.tc = (int)g.taps;
        p.strip_cap = pb; p.stage = stage; p.lds_bytes = lds;
        p.cl_pitch = pitch; p.cl_fpb = fpb;
        p.svec = svec ? 1 : 0;
        p.fvec = fvec ? 1 : 0;
        p.strip_items = svec ? vec_items : 0;
        p.fused_fast = fused_fast ? 1 : 0;
        p.fused_ipt = raw_items > kConvThreads ? 2 : 1;
        p.fast = fvec && svec && g.c % kRC == 0 && g.k % t.bm == 0 ? 1 : 0;
        const int64_t blocks = ((g.npix + t.bn - 1) / t.bn) * ((g.k + t.bm - 1) / t.bm);
        if (blocks >= 256) {
            best = p;
            best_blocks = blocks;
            break;
        }
        if (blocks > best_blocks) { best = p; best_blocks = blocks; }
    }
    if (best.kind == ConvPlan::kNone) return plan_conv_f32(g);
    // The fast kernels also have a 128 x 256 tile (8 waves of 64 x 64, two per
    // SIMD: half the filter copies per pixel).  It only fits one workgroup per
    // CU, as 128 x 128 does, so it is taken when it needs no more rounds of
    // workgroups over the CUs.
    const int64_t raw256 = raw_rows_bound(g, 256) * g.w;
    if (best.bm == 128 && best.bn == 128 &&
        (fused ? best.fused_fast && raw256 <= (int64_t)kConvThreads * kBf16FusedItems : best.fast)) {
        ConvPlan q = best;
        q.bn = 256;
        const int64_t run_vec = strip_capacity(g, 256, 4);
        const int64_t vec_items = 2 * ((run_vec + 3) / 4);
        const int64_t ext = cl_extent_bound(g, 256, pitch) + kBf16Spare;
        const int64_t pb = ext + mod16((int)((2 - ext) % 16));
        const int64_t stage = 16 * (pb + q.cl_fpb);
        const int64_t blocks = ((g.npix + 255) / 256) * (g.k / 128);
        if (vec_items <= (int64_t)kConvThreads * kStripVecItems && 2 * stage * 2 <= kConvLdsMaxBytes &&
            (blocks + 255) / 256 <= (best_blocks + 255) / 256) {
            q.strip_cap = pb;
            q.stage = stage;
            q.lds_bytes = 2 * stage * 2;
            q.strip_items = vec_items;
            q.fused_ipt = raw256 > kConvThreads ? 2 : 1;
            return q;
        }
    }
    return best;
}

ConvArgs conv_args_bf16(const Geometry& g, const ConvPlan& p, const void* src, const void* w,
                        float* y, bool fused) {
    ConvArgs a = make_conv_args(g, src, w, y, p.bm);
    a.rc = kRC;
    a.strip_cap = (int)p.strip_cap;
    a.stage = (int)p.stage;
    a.tc = p.tc;
    a.svec = (!fused && p.svec) ? 1 : 0;
    a.vchunk = 4;
    a.fvec = p.fvec;
    a.cl_pitch = (int)p.cl_pitch;
    a.cl_pb = (int)p.strip_cap;
    a.cl_fpb = (int)p.cl_fpb;
    a.div_ckmid = make_fastdiv((uint32_t)((((g.ho - 1) * g.row_len + g.used_len) + 3) >> 2));
    return a;
}

int bf16_strip_mode(const ConvPlan& p, bool fused) {
    return fused ? kStripFused : (p.svec ? kStripVec : kStripScalar);
}

// The fast kernels read the filter packed (packed_piece).
bool bf16_packed(const ConvPlan& p, bool fused) { return fused ? p.fused_fast != 0 : p.fast != 0; }

int64_t conv_scratch_bytes(const Geometry& g, bool fused) {
    if (plan_image_bf16(g, fused).ok) return g.k * g.c * g.taps * 2;
    if (plan_band_f32(g).ok || plan_band_small_c_f32(g).ok) return 0;   // read the filter as given
    const ConvPlan p = g.elem == 2 ? plan_conv_bf16(g, fused) : plan_conv_f32(g);
    if (p.kind == ConvPlan::kNone) return -1;
    if (p.kind == ConvPlan::kF32Lds) return filter_scratch_f32(g, p);
    return bf16_packed(p, fused) ? g.k * g.c * g.taps * 2 : 0;
}

const char* conv_kernel_name(const Geometry& g, bool fused) {
    if (plan_image_bf16(g, fused).ok) return "bf16_one_image";
    if (plan_band_f32(g).ok) return "f32_bands";
    if (plan_band_small_c_f32(g).ok) return "f32_bands_small_c";
    const ConvPlan p = g.elem == 2 ? plan_conv_bf16(g, fused) : plan_conv_f32(g);
    if (p.kind == ConvPlan::kNone) return "per_output";
    if (g.elem == 2) return p.kind == ConvPlan::kF32Lds ? "bf16_widened_tiles" : "bf16_tiles";
    return "f32_tiles";
}

int launch_conv_bf16(const Geometry& g, bool fused, const void* src, const void* w, void* scratch,
                     float* y, hipStream_t stream, char* err, size_t errlen) {
    const ImgPlan ip = plan_image_bf16(g, fused);
    if (ip.ok) return launch_conv_bf16_image(g, ip, fused, src, w, scratch, y, stream);
    const ConvPlan p = plan_conv_bf16(g, fused);
    if (p.kind == ConvPlan::kNone) return launch_conv_plain(g, fused, src, w, y, stream, err, errlen);
    if (p.kind == ConvPlan::kF32Lds)
        return launch_conv_f32_plan(g, p, fused, src, w, scratch, y, stream, err, errlen);
    ConvArgs a = conv_args_bf16(g, p, src, w, y, fused);
    const int64_t blocks = ((g.npix + p.bn - 1) / p.bn) * a.num_jtiles;
    if (blocks > 0x7fffffff) {
        snprintf(err, errlen, "conv: grid of %lld workgroups is too large", (long long)blocks);
        return -5;
    }
    const int smode = bf16_strip_mode(p, fused);
    if (bf16_packed(p, fused)) {
        // the filter, repacked for 16-byte copies, into the caller's scratch
        // (K*C*Fh*Fw*2 bytes)
        const int64_t nchunks = g.c / kRC;
        hipLaunchKernelGGL(pack_filter_bf16_kernel, dim3((unsigned)(g.k / kPackRows * nchunks)), dim3(256),
                           (size_t)kPackRows * kRC * g.taps * 2, stream, static_cast<const uint16_t*>(w),
                           static_cast<uint16_t*>(scratch), (int)g.c, (int)g.fh, (int)g.fw, p.bm, (int)nchunks);
        a.w = scratch;
    }
    if (p.fvec && g.fh == 3 && g.fw == 3) launch_tile<3, 3, true>(p, a, blocks, smode, stream);
    else if (p.fvec && g.fh == 3 && g.fw == 5) launch_tile<3, 5, true>(p, a, blocks, smode, stream);
    else if (p.fvec && g.fh == 1 && g.fw == 1) launch_tile<1, 1, true>(p, a, blocks, smode, stream);
    else launch_tile<0, 0, false>(p, a, blocks, smode, stream);
    return 0;
}

}  // namespace im2win
