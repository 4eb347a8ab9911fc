// fp32 im2win convolution on gfx950 matrix cores (Alg. 2 semantics).
//
// The convolution is an implicit GEMM  Y[j][p] = sum_kk F[j][kk] * Win[kk][p]
// over output channels j, output pixels p = (i, m, n) and the reduction index
// kk = (r, t), t = v*Fh + u.  Because the window tensor stores each window as
// the contiguous run [n*sw*Fh, n*sw*Fh + Fw*Fh) of row (i, r, m), the operand
// Win[(r, t)][p] is  strip_r[base(p) + t]: horizontally adjacent windows
// overlap inside one strip and are read from the same on-chip copy (the data
// reuse the paper builds its loop order around, Sec. III-B).
//
// Workgroup = 4 waves computing a BM (channels) x BN (pixels) tile of Y.
// Pixels are tiled in flattened (i, m, n) order, so a tile covers a handful
// of window-tensor rows, which for one channel are contiguous in memory
// (one run per image).  Per chunk of `rc` input channels the workgroup:
//   - copies those runs into LDS (unfused: from the window tensor; fused:
//     builds them from x, zero padding included, never touching HBM for Win),
//   - stages the filter chunk as F[kk][j] (kk in window order),
//   - runs v_mfma_f32_32x32x2f32: A = filter rows (32 channels), B = window
//     columns (32 pixels), so each accumulator register holds 32 consecutive
//     pixels of one output channel and the NCHW stores are coalesced.
#include "conv_common.h"

#include <algorithm>
#include <cstdio>

namespace im2win {
namespace {

// Input elements are fp32, or bf16 bit patterns widened to fp32 when staged
// (exact; the bf16 fallback path for problems whose channel-inner bf16 tiles
// do not fit in LDS).
__device__ inline float to_f32(float v) { return v; }
__device__ inline float to_f32(uint16_t v) { return __uint_as_float(uint32_t(v) << 16); }

// Copy (unfused) or build (fused) the strips of channels [r0, r0+rc_act).
template <typename TIn, bool FUSED>
__device__ inline void stage_strips(float* S, const ConvArgs& a, const TileRuns& tr, int r0,
                                    int rc_act) {
    for (int rc = 0; rc < rc_act; ++rc) {
        const int r = r0 + rc;
        for (int s = 0; s < tr.nseg; ++s) {
            const int len = tr.seg_len(s);
            const int i = tr.i0 + s;
            const int ma = tr.seg_m(s), qa = tr.seg_q(s);
            float* dst = S + rc * a.strip_cap + tr.seg_off(s);
            if (!FUSED) {
                const TIn* src = static_cast<const TIn*>(a.src) +
                                 (((int64_t)i * a.c + r) * a.ho + ma) * a.row_len + qa;
                for (int e = threadIdx.x; e < len; e += kConvThreads) dst[e] = to_f32(src[e]);
            } else {
                const TIn* plane = static_cast<const TIn*>(a.src) +
                                   ((int64_t)i * a.c + r) * a.h * a.w_in;
                int e = threadIdx.x;
                if (e >= len) continue;
                const int pos = qa + e;
                int row = (int)fast_div((uint32_t)pos, a.div_row);
                const int q = pos - row * a.row_len;
                int kcol = (int)fast_div((uint32_t)q, a.div_fh);
                int u = q - kcol * a.fh;
                for (; e < len; e += kConvThreads) {
                    const int yy = (ma + row) * a.sh + u - a.ph;
                    const int xx = kcol - a.pw;
                    float v = 0.0f;
                    if ((unsigned)yy < (unsigned)a.h && (unsigned)xx < (unsigned)a.w_in)
                        v = to_f32(plane[(int64_t)yy * a.w_in + xx]);
                    dst[e] = v;
                    u += a.d_u;
                    if (u >= a.fh) { u -= a.fh; ++kcol; }
                    kcol += a.d_k;
                    if (kcol >= a.wp) { kcol -= a.wp; ++row; }
                    row += a.d_row;
                }
            }
        }
    }
}

// F[kk][j] for kk = (r - r0)*T + v*Fh + u, zero outside the real filter.
template <typename TIn, int BM>
__device__ inline void stage_filter(float* F, const ConvArgs& a, int j0, int r0, int rc_act) {
    const int kreal = rc_act * a.taps;
    for (int idx = threadIdx.x; idx < BM * a.kpad; idx += kConvThreads) {
        const int jj = (int)fast_div((uint32_t)idx, a.div_kpad);
        const int nat = idx - jj * a.kpad;          // natural (r, u, v) order within the chunk
        const int j = j0 + jj;
        int kk = nat;
        float v = 0.0f;
        if (nat < kreal && j < a.k) {
            const int rl = (int)fast_div((uint32_t)nat, a.div_taps);
            const int tt = nat - rl * a.taps;
            const int u = (int)fast_div((uint32_t)tt, a.div_fw);
            const int vv = tt - u * a.fw;
            kk = rl * a.taps + vv * a.fh + u;
            v = to_f32(static_cast<const TIn*>(a.w)[((int64_t)j * a.c + r0) * a.taps + nat]);
        }
        F[kk * (BM + 1) + jj] = v;
    }
}

template <typename TIn, int BM, int BN, int TJ, int TP, bool FUSED>
__global__ __launch_bounds__(kConvThreads) void conv_f32_kernel(ConvArgs a) {
    static_assert((BM / TJ) * (BN / TP) == kConvThreads / 64, "4 waves per workgroup");
    constexpr int NJ = TJ / 32, NP = TP / 32;
    constexpr int WAVES_P = BN / TP;

    extern __shared__ __align__(16) unsigned char smem[];
    float* S = reinterpret_cast<float*>(smem);
    float* F = S + a.rc * a.strip_cap;
    float* Z = F + a.kpad * (BM + 1);   // one zero word for padded reduction slots

    const int jtile = blockIdx.x % a.num_jtiles;
    const int ptile = blockIdx.x / a.num_jtiles;
    const int j0 = jtile * BM;

    TileRuns tr;
    tr.init(ptile, BN, a);

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int wj = wave / WAVES_P, wp_ = wave % WAVES_P;
    const int l32 = lane & 31, kl = lane >> 5;

    // Per-lane pixel columns: strip offset of the window start and output offset.
    int pbase[NP];
    int64_t yoff[NP];
    bool pvalid[NP];
#pragma unroll
    for (int pb = 0; pb < NP; ++pb) {
        int p = tr.p0 + wp_ * TP + pb * 32 + l32;
        pvalid[pb] = p <= tr.plast;
        if (!pvalid[pb]) p = tr.p0;
        pbase[pb] = pixel_base(tr, a, p, &yoff[pb]);
    }
    int jrow[NJ];
#pragma unroll
    for (int jb = 0; jb < NJ; ++jb) jrow[jb] = wj * TJ + jb * 32 + l32;

    f32x16 acc[NJ][NP];
#pragma unroll
    for (int jb = 0; jb < NJ; ++jb)
#pragma unroll
        for (int pb = 0; pb < NP; ++pb)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[jb][pb][v] = 0.0f;

    if (threadIdx.x == 0) Z[0] = 0.0f;
    const int zero_off = (int)(Z - S);

    for (int r0 = 0; r0 < a.c; r0 += a.rc) {
        const int rc_act = min(a.rc, a.c - r0);
        __syncthreads();
        stage_strips<TIn, FUSED>(S, a, tr, r0, rc_act);
        stage_filter<TIn, BM>(F, a, j0, r0, rc_act);
        __syncthreads();

        const int kreal = rc_act * a.taps;
        const int ksteps = (kreal + 1) >> 1;
        int rck = 0, tk = kl;
        while (tk >= a.taps) { tk -= a.taps; ++rck; }
        for (int s = 0; s < ksteps; ++s) {
            const int kk = 2 * s + kl;
            const int koff = rck * a.strip_cap + tk;
            float av[NJ], bv[NP];
#pragma unroll
            for (int jb = 0; jb < NJ; ++jb) av[jb] = F[kk * (BM + 1) + jrow[jb]];
#pragma unroll
            for (int pb = 0; pb < NP; ++pb) bv[pb] = S[kk < kreal ? pbase[pb] + koff : zero_off];
#pragma unroll
            for (int jb = 0; jb < NJ; ++jb)
#pragma unroll
                for (int pb = 0; pb < NP; ++pb)
                    acc[jb][pb] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[jb], bv[pb], acc[jb][pb], 0, 0, 0);
            tk += 2;
            while (tk >= a.taps) { tk -= a.taps; ++rck; }
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

template <typename TIn, int BM, int BN, int TJ, int TP>
void launch_cfg(const ConvArgs& a, int64_t blocks, int64_t lds, bool fused, hipStream_t stream) {
    if (fused)
        hipLaunchKernelGGL((conv_f32_kernel<TIn, BM, BN, TJ, TP, true>), dim3((unsigned)blocks),
                           dim3(kConvThreads), (size_t)lds, stream, a);
    else
        hipLaunchKernelGGL((conv_f32_kernel<TIn, BM, BN, TJ, TP, false>), dim3((unsigned)blocks),
                           dim3(kConvThreads), (size_t)lds, stream, a);
}

template <typename TIn>
void launch_plan(const ConvPlan& p, const ConvArgs& a, int64_t blocks, bool fused,
                 hipStream_t stream) {
    if (p.bm == 64 && p.bn == 256) launch_cfg<TIn, 64, 256, 64, 64>(a, blocks, p.lds_bytes, fused, stream);
    else if (p.bm == 128) launch_cfg<TIn, 128, 128, 64, 64>(a, blocks, p.lds_bytes, fused, stream);
    else if (p.bn == 128) launch_cfg<TIn, 64, 128, 32, 64>(a, blocks, p.lds_bytes, fused, stream);
    else launch_cfg<TIn, 64, 64, 32, 32>(a, blocks, p.lds_bytes, fused, stream);
}

int64_t lds_bytes_f32(int bm, int rc, int64_t taps, int64_t strip_cap) {
    const int64_t kpad = (rc * taps + 1) & ~int64_t(1);
    return ((int64_t)rc * strip_cap + kpad * (bm + 1) + 4) * 4;
}

}  // namespace

// Tile candidates, preferred first; the first whose LDS fits is used, with
// the largest channel chunk that fits.  The window strips and the filter tile
// are held in fp32 whatever the input type.
ConvPlan plan_conv_f32(const Geometry& g) {
    const TileCfg cfgs_small_k[] = {{64, 256}, {64, 128}, {64, 64}};
    const TileCfg cfgs_large_k[] = {{128, 128}, {64, 128}, {64, 64}};
    const TileCfg* cfgs = g.k <= 64 ? cfgs_small_k : cfgs_large_k;
    ConvPlan p;
    for (int ci = 0; ci < 3; ++ci) {
        const int64_t cap = strip_bound(g, cfgs[ci].bn);
        for (int rc = 1; rc <= std::min<int64_t>(g.c, 32); ++rc) {
            const int64_t lds = lds_bytes_f32(cfgs[ci].bm, rc, g.taps, cap);
            if (lds > kConvLdsBudgetBytes) break;
            p.kind = ConvPlan::kF32Lds;
            p.bm = cfgs[ci].bm; p.bn = cfgs[ci].bn; p.rc = rc; p.tc = (int)g.taps;
            p.strip_cap = cap; p.lds_bytes = lds;
        }
        if (p.rc > 0) break;
    }
    return p;
}

ConvArgs conv_args_f32(const Geometry& g, const ConvPlan& p, const void* src, const void* w,
                       float* y) {
    ConvArgs a = make_conv_args(g, src, w, y, p.bm);
    a.rc = p.rc;
    a.strip_cap = (int)p.strip_cap;
    a.kpad = (p.rc * a.taps + 1) & ~1;
    a.div_kpad = make_fastdiv((uint32_t)a.kpad);
    return a;
}

int launch_conv_f32_plan(const Geometry& g, const ConvPlan& p, bool fused, const void* src,
                         const void* w, float* y, hipStream_t stream, char* err, size_t errlen) {
    const ConvArgs a = conv_args_f32(g, p, src, w, y);
    const int64_t blocks = ((g.npix + p.bn - 1) / p.bn) * a.num_jtiles;
    if (blocks > 0x7fffffff) {
        snprintf(err, errlen, "conv: grid of %lld workgroups is too large", (long long)blocks);
        return -5;
    }
    if (g.elem == 4) launch_plan<float>(p, a, blocks, fused, stream);
    else launch_plan<uint16_t>(p, a, blocks, fused, stream);
    return 0;
}

int launch_conv_f32(const Geometry& g, bool fused, const void* src, const void* w, float* y,
                    hipStream_t stream, char* err, size_t errlen) {
    const ConvPlan p = plan_conv_f32(g);
    if (p.rc == 0) {
        snprintf(err, errlen,
                 "conv: the window strips of one tile (row length %lld) do not fit in LDS; "
                 "this shape is not supported", (long long)g.row_len);
        return -5;
    }
    return launch_conv_f32_plan(g, p, fused, src, w, y, stream, err, errlen);
}

}  // namespace im2win
