// bf16 im2win convolution on gfx950 matrix cores, fp32 accumulation.
//
// Same implicit GEMM and pixel tiling as the fp32 kernel, with the reduction
// ordered tap-major: kk = (t, r) with t = v*Fh + u.  For each tap the matrix
// core contracts 16 input channels (v_mfma_f32_32x32x16_bf16: 8 consecutive
// reduction elements per lane), so the LDS holds the window strips with the
// channel innermost, S[pos][16], and a lane's operand for pixel p and tap t is
// the 16-byte vector S[base(p) + t][8h .. 8h+7].  Each strip position is
// still the window-tensor element at that row position: a window stays the
// contiguous run of positions [base(p), base(p) + Fw*Fh), shared by
// overlapping windows.  The filter is staged as F[t][j][16].
//
// Per chunk of 16 input channels the workgroup builds the strips once, then
// walks the taps in passes of `tc` taps (filter tiles of large filters do not
// fit in LDS at once).  Channels beyond C are zero in both operands.
#include "conv_common.h"

#include <cstdio>

namespace im2win {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kRC = 16;   // input channels per chunk (the MFMA reduction width)

struct alignas(16) U16x8 {
    uint16_t v[8];
};

template <bool FUSED>
__device__ inline void stage_strips(uint16_t* S, const ConvArgs& a, const TileRuns& tr, int r0) {
    const uint16_t* src = static_cast<const uint16_t*>(a.src);
    const int nseg = tr.nseg, i0 = tr.i0, len0 = tr.len0, len_mid = tr.len_mid,
              len_last = tr.len_last, m0 = tr.m0, qa0 = tr.qa0, d_first = tr.d_first,
              d_second = tr.d_second, d_stride = tr.d_stride;
    for (int grp = 0; grp < 2; ++grp) {
        const int rbase = r0 + 8 * grp;
        for (int s = 0; s < nseg; ++s) {
            const SegRun sr = seg_run(s, nseg, len0, len_mid, len_last, m0, qa0, d_first, d_second, d_stride);
            const int len = sr.len;
            const int i = i0 + s;
            const int ma = sr.m, qa = sr.q;
            uint16_t* dst = S + (int64_t)sr.off * kRC + 8 * grp;
            int e = threadIdx.x;
            if (e >= len) continue;
            if (!FUSED) {
                const int64_t plane_len = (int64_t)a.ho * a.row_len;
                const uint16_t* run = src + (((int64_t)i * a.c + rbase) * a.ho + ma) * a.row_len + qa;
                for (; e < len; e += kConvThreads) {
                    U16x8 v;
#pragma unroll
                    for (int ch = 0; ch < 8; ++ch)
                        v.v[ch] = (rbase + ch < a.c) ? run[ch * plane_len + e] : uint16_t(0);
                    *reinterpret_cast<U16x8*>(dst + (int64_t)e * kRC) = v;
                }
            } else {
                const int64_t plane_len = (int64_t)a.h * a.w_in;
                const uint16_t* planes = src + ((int64_t)i * a.c + rbase) * plane_len;
                const int pos = qa + e;
                int row = (int)fast_div((uint32_t)pos, a.div_row);
                const int q = pos - row * a.row_len;
                int kcol = (int)fast_div((uint32_t)q, a.div_fh);
                int u = q - kcol * a.fh;
                for (; e < len; e += kConvThreads) {
                    const int yy = (ma + row) * a.sh + u - a.ph;
                    const int xx = kcol - a.pw;
                    const bool inb = (unsigned)yy < (unsigned)a.h && (unsigned)xx < (unsigned)a.w_in;
                    const int64_t off = (int64_t)yy * a.w_in + xx;
                    U16x8 v;
#pragma unroll
                    for (int ch = 0; ch < 8; ++ch)
                        v.v[ch] = (inb && rbase + ch < a.c) ? planes[ch * plane_len + off] : uint16_t(0);
                    *reinterpret_cast<U16x8*>(dst + (int64_t)e * kRC) = v;
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

// F[tl][j][16] for taps t0 + tl, channels r0 .. r0+15 (zero outside the filter).
template <int BM>
__device__ inline void stage_filter(uint16_t* F, const ConvArgs& a, int j0, int r0, int t0,
                                    int tc_act) {
    const uint16_t* w = static_cast<const uint16_t*>(a.w);
    const int tasks = BM * a.tc * 2;
    for (int idx = threadIdx.x; idx < tasks; idx += kConvThreads) {
        const int jj = (int)fast_div((uint32_t)idx, a.div_tc2);   // div by 2*tc
        const int rem = idx - jj * 2 * a.tc;
        const int tl = rem >> 1, grp = rem & 1;
        U16x8 v;
        const int j = j0 + jj;
        if (tl < tc_act && j < a.k) {
            const int t = t0 + tl;
            const int vv = (int)fast_div((uint32_t)t, a.div_fh);
            const int u = t - vv * a.fh;
            const int rbase = r0 + 8 * grp;
            const uint16_t* wp = w + ((int64_t)j * a.c + rbase) * a.taps + u * a.fw + vv;
#pragma unroll
            for (int ch = 0; ch < 8; ++ch)
                v.v[ch] = (rbase + ch < a.c) ? wp[ch * a.taps] : uint16_t(0);
        } else {
#pragma unroll
            for (int ch = 0; ch < 8; ++ch) v.v[ch] = 0;
        }
        if (tl < tc_act)
            *reinterpret_cast<U16x8*>(F + ((int64_t)(tl * BM + jj) * kRC + 8 * grp)) = v;
    }
}

__device__ inline bf16x8 lds_frag(const uint16_t* p) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const U16x8*>(p));
}

template <int BM, int BN, int TJ, int TP, bool FUSED>
__global__ __launch_bounds__(kConvThreads) void conv_bf16_kernel(ConvArgs a) {
    static_assert((BM / TJ) * (BN / TP) == kConvThreads / 64, "4 waves per workgroup");
    constexpr int NJ = TJ / 32, NP = TP / 32;
    constexpr int WAVES_P = BN / TP;

    extern __shared__ __align__(16) unsigned char smem[];
    uint16_t* S = reinterpret_cast<uint16_t*>(smem);
    uint16_t* F = S + (int64_t)a.strip_cap * kRC;

    const int jtile = blockIdx.x % a.num_jtiles;
    const int ptile = blockIdx.x / a.num_jtiles;
    const int j0 = jtile * BM;

    TileRuns tr;
    tr.init(ptile, BN, a);

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int wj = wave / WAVES_P, wp_ = wave % WAVES_P;
    const int l32 = lane & 31, kl = lane >> 5;

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

    for (int r0 = 0; r0 < a.c; r0 += kRC) {
        __syncthreads();
        stage_strips<FUSED>(S, a, tr, r0);
        for (int t0 = 0; t0 < a.taps; t0 += a.tc) {
            const int tc_act = min(a.tc, a.taps - t0);
            if (t0 > 0) __syncthreads();
            stage_filter<BM>(F, a, j0, r0, t0, tc_act);
            __syncthreads();
            for (int tl = 0; tl < tc_act; ++tl) {
                const int t = t0 + tl;
                bf16x8 av[NJ], bv[NP];
#pragma unroll
                for (int jb = 0; jb < NJ; ++jb)
                    av[jb] = lds_frag(F + (int64_t)(tl * BM + jrow[jb]) * kRC + 8 * kl);
#pragma unroll
                for (int pb = 0; pb < NP; ++pb)
                    bv[pb] = lds_frag(S + (int64_t)(pbase[pb] + t) * kRC + 8 * kl);
#pragma unroll
                for (int jb = 0; jb < NJ; ++jb)
#pragma unroll
                    for (int pb = 0; pb < NP; ++pb)
                        acc[jb][pb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[jb], bv[pb], acc[jb][pb], 0, 0, 0);
            }
        }
    }

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

template <int BM, int BN, int TJ, int TP>
void launch_cfg(const ConvArgs& a, int64_t blocks, int64_t lds, bool fused, hipStream_t stream) {
    if (fused)
        hipLaunchKernelGGL((conv_bf16_kernel<BM, BN, TJ, TP, true>), dim3((unsigned)blocks),
                           dim3(kConvThreads), (size_t)lds, stream, a);
    else
        hipLaunchKernelGGL((conv_bf16_kernel<BM, BN, TJ, TP, false>), dim3((unsigned)blocks),
                           dim3(kConvThreads), (size_t)lds, stream, a);
}

}  // namespace

// Tile candidates, preferred first; the first whose LDS fits is used, with
// the most filter taps per pass that fit.  When none fits (large windows with
// little overlap), the bf16 problem runs on the fp32-strip kernel instead.
ConvPlan plan_conv_bf16(const Geometry& g) {
    const TileCfg cfgs_small_k[] = {{64, 256}, {64, 128}, {64, 64}};
    const TileCfg cfgs_large_k[] = {{128, 128}, {64, 128}, {64, 64}};
    const TileCfg* cfgs = g.k <= 64 ? cfgs_small_k : cfgs_large_k;
    ConvPlan p;
    for (int ci = 0; ci < 3; ++ci) {
        const int64_t cap = strip_bound(g, cfgs[ci].bn);
        for (int tc = 1; tc <= g.taps; ++tc) {
            const int64_t lds = (cap + (int64_t)tc * cfgs[ci].bm) * kRC * 2;
            if (lds > kConvLdsBudgetBytes) break;
            p.kind = ConvPlan::kBf16Lds;
            p.bm = cfgs[ci].bm; p.bn = cfgs[ci].bn; p.rc = kRC; p.tc = tc;
            p.strip_cap = cap; p.lds_bytes = lds;
        }
        if (p.tc > 0) return p;
    }
    return plan_conv_f32(g);
}

ConvArgs conv_args_bf16(const Geometry& g, const ConvPlan& p, const void* src, const void* w,
                        float* y) {
    ConvArgs a = make_conv_args(g, src, w, y, p.bm);
    a.rc = kRC;
    a.strip_cap = (int)p.strip_cap;
    a.tc = p.tc;
    a.div_tc2 = make_fastdiv((uint32_t)(2 * p.tc));
    return a;
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
    const ConvArgs a = conv_args_bf16(g, p, src, w, y);
    const int64_t blocks = ((g.npix + p.bn - 1) / p.bn) * a.num_jtiles;
    if (blocks > 0x7fffffff) {
        snprintf(err, errlen, "conv: grid of %lld workgroups is too large", (long long)blocks);
        return -5;
    }
    if (p.bm == 64 && p.bn == 256) launch_cfg<64, 256, 64, 64>(a, blocks, p.lds_bytes, fused, stream);
    else if (p.bm == 128) launch_cfg<128, 128, 64, 64>(a, blocks, p.lds_bytes, fused, stream);
    else if (p.bn == 128) launch_cfg<64, 128, 32, 64>(a, blocks, p.lds_bytes, fused, stream);
    else launch_cfg<64, 64, 32, 32>(a, blocks, p.lds_bytes, fused, stream);
    return 0;
}

}  // namespace im2win
