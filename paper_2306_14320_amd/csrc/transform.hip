// im2win transformation on gfx950 (Alg. 1 / Eq. 2 with zero padding):
//   ws[i][r][m][k*Fh + u] = x[i][r][m*sh + u - ph][k - pw]   (0 outside x)
//
// Pure data movement, bound by HBM bandwidth.  Each workgroup owns one
// contiguous run of window-tensor rows: either a tile of `tm` rows of one
// image plane (large planes) or `g` whole image planes (small planes).  It
//   1. clears the run in LDS (padding positions stay zero),
//   2. reads the input rows the run uses once, coalesced, eight loads in
//      flight per thread, and writes every element to the ceil(Fh/sh)
//      positions of the run that hold it (the Fh/sh-fold duplication of the
//      window tensor happens on chip),
//   3. copies the finished run to global memory with 16-byte LDS reads and
//      16-byte stores in address order.
// Elements move as raw bits (uint32 for fp32, uint16 for bf16): the copy is
// exact.
#include "common.h"

#include <algorithm>
#include <cstdio>
#include <type_traits>

namespace im2win {
namespace {

constexpr int kThreads = 256;
constexpr int kOutTargetBytes = 24 * 1024;   // output bytes per workgroup (target)
constexpr int kLdsBudgetBytes = 64 * 1024;   // LDS per workgroup (cap)

template <typename T, int V>
struct alignas(V * sizeof(T)) Vec {
    T v[V];
};

// TRIM: the rows are narrower than the input reaches (trimmed layout), so
// input columns past the row's last window are skipped.
template <typename T, int V, bool TRIM>
__global__ __launch_bounds__(kThreads) void transform_lds_kernel(XformArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    T* lds = reinterpret_cast<T*>(smem);
    const T* __restrict__ x = static_cast<const T*>(a.x);
    T* __restrict__ ws = static_cast<T*>(a.ws);

    XformBlock blk;
    blk.init(blockIdx.x, a);
    const int span = blk.shift + blk.olen;             // LDS elements in use
    const int nvec_lds = (span + V - 1) / V;

    // 1. clear
    Vec<T, V> zero;
#pragma unroll
    for (int j = 0; j < V; ++j) zero.v[j] = T(0);
    for (int i = threadIdx.x; i < nvec_lds; i += kThreads) reinterpret_cast<Vec<T, V>*>(lds)[i] = zero;
    __syncthreads();

    // 2. scatter the input rows [y_lo, y_lo + nrin) of each plane.  When the
    // footprint of a plane starts and ends on 16-byte boundaries each thread
    // loads whole 16-byte vectors (V elements), else single elements; either
    // way eight loads are in flight per thread before any value is placed.
    const int per_plane = blk.nrin * a.w;
    const int total = blk.nplanes * per_plane;
    const int64_t plane_len = (int64_t)a.h * a.w;
    const bool vec_in = a.vec_in && ((int64_t)blk.y_lo * a.w) % V == 0;
    // Element f of the footprint and the VV after it lie in one input row
    // (VV divides W): the row's destinations are decoded once, and element t
    // goes to the first one's LDS index + t*Fh in each destination row.
    auto place = [&](const T* v, int f, auto vv) {
        constexpr int VV = decltype(vv)::value;
        const int pj = a.g > 1 ? (int)fast_div((uint32_t)f, a.div_plane) : 0;
        const int rem = f - pj * per_plane;
        const int r = (int)fast_div((uint32_t)rem, a.div_w);
        const int yy = blk.y_lo + r, xx = rem - r * a.w;
        int mf, ml;
        blk.rows_of(yy, a, &mf, &ml);
        for (int m = mf; m <= ml; ++m) {
            T* d = lds + blk.lds_index(pj, m, xx + a.pw, yy + a.ph - m * a.sh, a);
#pragma unroll
            for (int t = 0; t < VV; ++t)
                if (!TRIM || xx + a.pw + t < a.wp) d[t * a.fh] = v[t];
        }
    };
    // footprint vectors of VV elements: plane starts, row y_lo and per_plane
    // are multiples of VV (VV divides W)
    auto vec_pass = [&](auto vv) {
        constexpr int VV = decltype(vv)::value;
        typedef Vec<T, VV> VT;
        const int nv = total / VV;
        for (int i0 = threadIdx.x; i0 < nv; i0 += 8 * kThreads) {
            VT v[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int i = i0 + j * kThreads;
                const int f = i * VV;
                const int pj = a.g > 1 ? (int)fast_div((uint32_t)f, a.div_plane) : 0;
                const int64_t src = (blk.plane0 + pj) * plane_len + (int64_t)blk.y_lo * a.w + (f - pj * per_plane);
                if (i < nv) v[j] = *reinterpret_cast<const VT*>(x + src);
            }
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int i = i0 + j * kThreads;
                if (i < nv) place(v[j].v, i * VV, vv);
            }
        }
    };
    if (vec_in) {
        vec_pass(std::integral_constant<int, V>());
    } else if (V > 2 && a.w % 2 == 0) {
        vec_pass(std::integral_constant<int, 2>());
    } else {
        for (int f0 = threadIdx.x; f0 < total; f0 += 8 * kThreads) {
            T v[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int f = f0 + j * kThreads;
                const int pj = a.g > 1 ? (int)fast_div((uint32_t)f, a.div_plane) : 0;
                const int64_t src = (blk.plane0 + pj) * plane_len + (int64_t)blk.y_lo * a.w + (f - pj * per_plane);
                v[j] = f < total ? x[src] : T(0);
            }
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (f0 + j * kThreads < total) place(&v[j], f0 + j * kThreads, std::integral_constant<int, 1>());
        }
    }
    __syncthreads();

    // 3. copy out; LDS index i is global element obase - shift + i
    const int64_t gbase = blk.obase - blk.shift;
    const int first_vec = blk.shift ? 1 : 0;
    const int last_vec = span / V;                      // vectors [first_vec, last_vec) are whole
    // (plain stores: the convolution that follows reads the window tensor
    // back, and finds much of it still in the caches)
    for (int i = first_vec + threadIdx.x; i < last_vec; i += kThreads)
        *reinterpret_cast<Vec<T, V>*>(ws + gbase + (int64_t)i * V) =
            reinterpret_cast<const Vec<T, V>*>(lds)[i];
    // partial head (before the first whole vector) and tail
    const int head_end = min(first_vec ? V : 0, span);
    for (int i = blk.shift + threadIdx.x; i < head_end; i += kThreads) ws[gbase + i] = lds[i];
    for (int i = max(last_vec * V, head_end) + threadIdx.x; i < span; i += kThreads)
        ws[gbase + i] = lds[i];
}

// Fallback for rows too long to build in LDS: one workgroup per
// window-tensor row, reading x directly (loads stay coalesced along k).
template <typename T>
__global__ __launch_bounds__(kThreads) void transform_direct_kernel(XformArgs a, int64_t nrows_total) {
    const T* __restrict__ x = static_cast<const T*>(a.x);
    T* __restrict__ ws = static_cast<T*>(a.ws);
    for (int64_t row = blockIdx.x; row < nrows_total; row += gridDim.x) {
        const int64_t plane = row / a.ho;
        const int m = (int)(row - plane * a.ho);
        T* dst = ws + row * a.row_len;
        for (int u = 0; u < a.fh; ++u) {
            const int yy = m * a.sh + u - a.ph;
            const bool row_ok = (unsigned)yy < (unsigned)a.h;
            const T* src = x + (plane * a.h + (row_ok ? yy : 0)) * (int64_t)a.w;
            for (int k = threadIdx.x; k < a.wp; k += kThreads) {
                const int xx = k - a.pw;
                dst[(int64_t)k * a.fh + u] =
                    (row_ok && (unsigned)xx < (unsigned)a.w) ? src[xx] : T(0);
            }
        }
    }
}

template <typename T, int V>
void launch(const XformArgs& a, const XformPlan& p, int64_t nrows_total, bool trim,
            hipStream_t stream) {
    if (p.use_lds && trim)
        hipLaunchKernelGGL((transform_lds_kernel<T, V, true>), dim3((unsigned)p.blocks), dim3(kThreads),
                           (size_t)p.lds_bytes, stream, a);
    else if (p.use_lds)
        hipLaunchKernelGGL((transform_lds_kernel<T, V, false>), dim3((unsigned)p.blocks), dim3(kThreads),
                           (size_t)p.lds_bytes, stream, a);
    else
        hipLaunchKernelGGL((transform_direct_kernel<T>), dim3((unsigned)p.blocks), dim3(kThreads),
                           0, stream, a, nrows_total);
}

}  // namespace

// Work split of the transformation (chosen on the host, replayed by the plan
// checker with the same arithmetic): about kOutTargetBytes of output per
// workgroup, the whole run held in LDS.
XformPlan plan_transform(const Geometry& g) {
    XformPlan p;
    const int64_t e = g.elem;
    const int64_t vec = 16 / e;
    const int64_t nc = g.n * g.c;
    const int64_t row_bytes = g.row_len * e;
    const int64_t plane_out = g.ho * row_bytes;
    int64_t tm, gp;
    // the split is balanced: the last tile of a plane (or the last group of
    // planes) is as large as the others, up to one row (plane)
    if (plane_out >= kOutTargetBytes / 2) {
        gp = 1;
        tm = std::max<int64_t>(1, std::min<int64_t>(g.ho, kOutTargetBytes / row_bytes));
        const int64_t tiles = (g.ho + tm - 1) / tm;
        tm = (g.ho + tiles - 1) / tiles;
    } else {
        tm = g.ho;
        gp = std::max<int64_t>(1, std::min<int64_t>(nc, kOutTargetBytes / plane_out));
        const int64_t groups = (nc + gp - 1) / gp;
        gp = (nc + groups - 1) / groups;
    }
    p.lds_bytes = (gp * tm * g.row_len + 2 * vec) * e;
    // the LDS kernel indexes a workgroup's run and footprint with 32-bit integers
    p.use_lds = p.lds_bytes <= kLdsBudgetBytes && gp * tm * g.row_len < (int64_t(1) << 30) &&
                gp * g.h * g.w < (int64_t(1) << 30);
    if (p.use_lds) {
        p.g = gp;
        p.tm = tm;
        p.tiles_per_plane = (g.ho + tm - 1) / tm;
        p.blocks = ((nc + gp - 1) / gp) * p.tiles_per_plane;
    } else {
        p.g = 1;
        p.tm = 1;
        p.tiles_per_plane = 1;
        p.lds_bytes = 0;
        p.blocks = std::min<int64_t>(nc * g.ho, 65536);
    }
    return p;
}

XformArgs transform_args(const Geometry& g, const XformPlan& p, const void* x, void* ws) {
    XformArgs a;
    a.x = x;
    a.ws = ws;
    a.nc = g.n * g.c;
    a.h = (int)g.h;
    a.w = (int)g.w;
    a.ho = (int)g.ho;
    a.wp = (int)g.wp;
    a.fh = (int)g.fh;
    a.sh = (int)g.sh;
    a.ph = (int)g.ph;
    a.pw = (int)g.pw;
    a.row_len = (int)g.row_len;
    a.g = (int)p.g;
    a.tm = (int)p.tm;
    a.tiles_per_plane = (int)p.tiles_per_plane;
    a.vec = 16 / g.elem;
    a.vec_in = ((g.h * g.w) % a.vec == 0 && g.w % a.vec == 0) ? 1 : 0;
    // with several planes per workgroup (tm == ho) every workgroup uses the
    // same input rows of each plane: [max(0, -ph), min(h, (ho-1)*sh - ph + fh))
    const int64_t rows = std::min<int64_t>(g.h, (g.ho - 1) * g.sh - g.ph + g.fh) - std::max<int64_t>(0, -g.ph);
    a.div_plane = make_fastdiv((uint32_t)std::max<int64_t>(1, std::min<int64_t>(rows * g.w, 0x7fffffff)));
    a.div_w = make_fastdiv((uint32_t)a.w);
    a.div_sh = make_fastdiv((uint32_t)a.sh);
    return a;
}

int launch_transform(const Geometry& g, const void* x, void* ws, hipStream_t stream, char* err,
                     size_t errlen) {
    const XformPlan p = plan_transform(g);
    if (p.blocks > 0x7fffffff) {
        snprintf(err, errlen, "transform: grid of %lld workgroups is too large", (long long)p.blocks);
        return -5;
    }
    const XformArgs a = transform_args(g, p, x, ws);
    const bool trim = g.w + g.pw > g.wp;   // some input columns lie past a row's end
    if (g.elem == 4) launch<uint32_t, 4>(a, p, g.n * g.c * g.ho, trim, stream);
    else launch<uint16_t, 8>(a, p, g.n * g.c * g.ho, trim, stream);
    return 0;
}

}  // namespace im2win
