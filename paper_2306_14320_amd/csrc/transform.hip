// im2win transformation on gfx950 (Alg. 1 / Eq. 2 with zero padding):
//   ws[i][r][m][k*Fh + u] = x[i][r][m*sh + u - ph][k - pw]   (0 outside x)
//
// Pure data movement, bound by HBM bandwidth.  Each workgroup owns one
// contiguous run of window-tensor rows: either a tile of `tm` rows of one
// image plane (large planes) or `g` whole image planes (small planes).  It
//   1. copies the input rows that run needs into LDS with coalesced loads
//      (rows of one plane are contiguous in x, so this is one linear copy),
//   2. writes its output run with 16-byte stores in address order, reading the
//      column-major strip values back from LDS.
// Every input element is read from HBM once per workgroup; the Fh/sh-fold
// duplication of the window tensor happens on chip.  Elements are moved as
// raw bits (uint32 for fp32, uint16 for bf16), so the copy is exact.
#include "common.h"

#include <algorithm>
#include <cstdio>

namespace im2win {
namespace {

constexpr int kThreads = 256;
constexpr int kOutTargetBytes = 32 * 1024;   // output bytes per workgroup (target)
constexpr int kLdsBudgetBytes = 48 * 1024;   // LDS per workgroup (cap)

template <typename T, int V>
struct alignas(16) Vec {
    T v[V];
};

template <typename T>
__device__ inline void stage_rows(T* lds, const T* __restrict__ x, const XformArgs& a,
                                  int64_t plane0, int nplanes, int y_lo, int nrin) {
    const int per_plane = nrin * a.w;
    if (nrin == a.h) {
        // whole planes: one contiguous run of nplanes*H*W elements
        const T* src = x + plane0 * (int64_t)a.h * a.w;
        const int total = nplanes * per_plane;
        for (int e = threadIdx.x; e < total; e += kThreads) lds[e] = src[e];
    } else {
        for (int p = 0; p < nplanes; ++p) {
            const T* src = x + ((plane0 + p) * (int64_t)a.h + y_lo) * a.w;
            T* dst = lds + p * per_plane;
            for (int e = threadIdx.x; e < per_plane; e += kThreads) dst[e] = src[e];
        }
    }
}

template <typename T>
__device__ inline T fetch(const T* lds, const Cursor& c, const XformArgs& a, const XformBlock& b) {
    const int yy = (b.m0 + c.mrel) * a.sh + c.u - a.ph;
    const int xx = c.k - a.pw;
    if ((unsigned)yy < (unsigned)a.h && (unsigned)xx < (unsigned)a.w)
        return lds[b.lds_index(c.plane, yy, xx, a.w)];
    return T(0);
}

template <typename T, int V>
__global__ __launch_bounds__(kThreads) void transform_lds_kernel(XformArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    T* lds = reinterpret_cast<T*>(smem);
    const T* __restrict__ x = static_cast<const T*>(a.x);
    T* __restrict__ ws = static_cast<T*>(a.ws);

    XformBlock blk;
    blk.init(blockIdx.x, a);
    stage_rows<T>(lds, x, a, blk.plane0, blk.nplanes, blk.y_lo, blk.nrin);
    __syncthreads();

    // This workgroup's output: one contiguous run [obase, obase + olen).
    const int64_t obase = blk.obase;
    const int olen = blk.olen;
    const int head = (int)min<int64_t>((V - (obase % V)) % V, olen);
    const int nvec = (olen - head) / V;
    const int tail0 = head + nvec * V;

    for (int vi = threadIdx.x; vi < nvec; vi += kThreads) {
        const int e0 = head + vi * V;
        Cursor c = locate(e0, a);
        Vec<T, V> out;
#pragma unroll
        for (int j = 0; j < V; ++j) {
            out.v[j] = fetch<T>(lds, c, a, blk);
            advance(c, a);
        }
        *reinterpret_cast<Vec<T, V>*>(ws + obase + e0) = out;
    }
    // unaligned head and tail, one element per thread
    const int nscalar = head + (olen - tail0);
    for (int s = threadIdx.x; s < nscalar; s += kThreads) {
        const int e = (s < head) ? s : tail0 + (s - head);
        Cursor c = locate(e, a);
        ws[obase + e] = fetch<T>(lds, c, a, blk);
    }
}

// Fallback for input rows too wide to stage in LDS: one workgroup per
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
void launch(const XformArgs& a, const XformPlan& p, int64_t nrows_total, hipStream_t stream) {
    if (p.use_lds)
        hipLaunchKernelGGL((transform_lds_kernel<T, V>), dim3((unsigned)p.blocks), dim3(kThreads),
                           (size_t)p.lds_bytes, stream, a);
    else
        hipLaunchKernelGGL((transform_direct_kernel<T>), dim3((unsigned)p.blocks), dim3(kThreads),
                           0, stream, a, nrows_total);
}

}  // namespace

// Work split of the transformation (chosen on the host, checked by the plan
// checker with the same arithmetic).
XformPlan plan_transform(const Geometry& g) {
    XformPlan p;
    const int64_t e = g.elem;
    const int64_t nc = g.n * g.c;
    const int64_t row_bytes = g.row_len * e;
    const int64_t plane_out = g.ho * row_bytes;
    auto rows_in = [&](int64_t tm) { return std::min<int64_t>(g.h, (tm - 1) * g.sh + g.fh); };
    int64_t tm, gp;
    if (plane_out >= kOutTargetBytes / 2) {
        gp = 1;
        tm = std::max<int64_t>(1, std::min<int64_t>(g.ho, kOutTargetBytes / row_bytes));
        while (tm > 1 && rows_in(tm) * g.w * e > kLdsBudgetBytes) --tm;
    } else {
        tm = g.ho;
        gp = std::max<int64_t>(1, std::min<int64_t>(nc, kOutTargetBytes / plane_out));
        while (gp > 1 && gp * rows_in(tm) * g.w * e > kLdsBudgetBytes) --gp;
    }
    p.lds_bytes = gp * rows_in(tm) * g.w * e;
    // the LDS path indexes a workgroup's output run with 32-bit integers
    p.use_lds = p.lds_bytes <= kLdsBudgetBytes && gp * tm * g.row_len < (int64_t(1) << 30);
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
    a.div_row = make_fastdiv((uint32_t)a.row_len);
    a.div_fh = make_fastdiv((uint32_t)a.fh);
    a.div_tm = make_fastdiv((uint32_t)a.tm);
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
    if (g.elem == 4) launch<uint32_t, 4>(a, p, g.n * g.c * g.ho, stream);
    else launch<uint16_t, 8>(a, p, g.n * g.c * g.ho, stream);
    return 0;
}

}  // namespace im2win
