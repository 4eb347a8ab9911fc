// The im2win convolution for shapes whose window strips no LDS tile of the
// matrix-core kernels can hold (very long window-tensor rows with few output
// columns).  One thread per output element reads its window straight from
// the window tensor: the window of output (m, n) in channel r is the run
// [n*sw*Fh, (n*sw + Fw)*Fh) of row (i, r, m), tap (u, v) at offset v*Fh + u
// (Alg. 2 with the window offset in input columns).  The fused variant reads
// the same elements from x, zero where they fall in the padding.  fp32
// products and sums, in the order channel, filter column, filter row.
#include <algorithm>

#include "common.h"

namespace im2win {
namespace {

struct PlainArgs {
    const void* src;        // window tensor, or x (fused)
    const void* w;          // K x C x Fh x Fw
    float* y;               // N x K x Ho x Wo
    int64_t total;          // N*K*Ho*Wo
    int64_t row_len;        // Wr*Fh
    int c, h, w_in, k, fh, fw, sh, sw, ph, pw, ho, wo;
};

__device__ inline float load_f(const float* p, int64_t i) { return p[i]; }
__device__ inline float load_f(const uint16_t* p, int64_t i) {
    return __uint_as_float(uint32_t(p[i]) << 16);   // bf16 -> fp32 is exact
}

template <typename T, bool FUSED>
__global__ __launch_bounds__(256) void conv_plain_kernel(PlainArgs a) {
    const T* src = static_cast<const T*>(a.src);
    const T* w = static_cast<const T*>(a.w);
    const int64_t step = (int64_t)gridDim.x * blockDim.x;
    for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < a.total; o += step) {
        int64_t t = o;
        const int n = (int)(t % a.wo); t /= a.wo;
        const int m = (int)(t % a.ho); t /= a.ho;
        const int j = (int)(t % a.k);
        const int64_t i = t / a.k;
        float acc = 0.0f;
        for (int r = 0; r < a.c; ++r) {
            const int64_t wbase = ((int64_t)j * a.c + r) * a.fh * a.fw;
            if (!FUSED) {
                // row (i, r, m) of the window tensor, window of column n
                const int64_t win = (((i * a.c + r) * a.ho) + m) * a.row_len + (int64_t)n * a.sw * a.fh;
                for (int v = 0; v < a.fw; ++v)
                    for (int u = 0; u < a.fh; ++u)
                        acc = fmaf(load_f(src, win + (int64_t)v * a.fh + u), load_f(w, wbase + (int64_t)u * a.fw + v), acc);
            } else {
                const int64_t plane = (i * a.c + r) * a.h * (int64_t)a.w_in;
                for (int v = 0; v < a.fw; ++v) {
                    const int xx = n * a.sw + v - a.pw;
                    for (int u = 0; u < a.fh; ++u) {
                        const int yy = m * a.sh + u - a.ph;
                        const float xv = (xx >= 0 && xx < a.w_in && yy >= 0 && yy < a.h)
                                             ? load_f(src, plane + (int64_t)yy * a.w_in + xx) : 0.0f;
                        acc = fmaf(xv, load_f(w, wbase + (int64_t)u * a.fw + v), acc);
                    }
                }
            }
        }
        a.y[o] = acc;
    }
}

}  // namespace

int launch_conv_plain(const Geometry& g, bool fused, const void* src, const void* w, float* y,
                      hipStream_t stream, char* err, size_t errlen) {
    PlainArgs a;
    a.src = src;
    a.w = w;
    a.y = y;
    a.total = g.npix * g.k;
    a.row_len = g.row_len;
    a.c = (int)g.c; a.h = (int)g.h; a.w_in = (int)g.w; a.k = (int)g.k;
    a.fh = (int)g.fh; a.fw = (int)g.fw; a.sh = (int)g.sh; a.sw = (int)g.sw;
    a.ph = (int)g.ph; a.pw = (int)g.pw; a.ho = (int)g.ho; a.wo = (int)g.wo;
    // a grid-stride loop covers any size
    const int64_t blocks = std::min<int64_t>((a.total + 255) / 256, int64_t(1) << 20);
    if (g.elem == 4)
        hipLaunchKernelGGL((fused ? conv_plain_kernel<float, true> : conv_plain_kernel<float, false>),
                           dim3((unsigned)blocks), dim3(256), 0, stream, a);
    else
        hipLaunchKernelGGL((fused ? conv_plain_kernel<uint16_t, true> : conv_plain_kernel<uint16_t, false>),
                           dim3((unsigned)blocks), dim3(256), 0, stream, a);
    (void)err;
    (void)errlen;
    return 0;
}

}  // namespace im2win
