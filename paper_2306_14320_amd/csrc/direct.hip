// Comparison baseline: direct convolution with no data transformation
// (Eq. 1; the paper's Sec. IV-B compares im2win against a direct
// convolution of this kind).  One thread per output element, input and filter
// read straight from global memory, fp32 accumulation in the order of Eq. 1
// (channel, then filter row, then filter column).  It is a timing and memory
// baseline: the im2win path never calls it.
#include <algorithm>

#include "direct.h"

namespace im2win {
namespace {

struct DirectArgs {
    const void* x;
    const void* w;
    float* y;
    int64_t total;          // N*K*Ho*Wo
    int c, h, w_in, k, fh, fw, sh, sw, ph, pw, ho, wo;
};

__device__ inline float load_f(const float* p, int64_t i) { return p[i]; }
__device__ inline float load_f(const uint16_t* p, int64_t i) {
    return __uint_as_float(uint32_t(p[i]) << 16);   // bf16 -> fp32 is exact
}

template <typename T>
__global__ __launch_bounds__(256) void direct_conv_kernel(DirectArgs a) {
    const T* x = static_cast<const T*>(a.x);
    const T* w = static_cast<const T*>(a.w);
    const int64_t step = (int64_t)gridDim.x * blockDim.x;
    for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < a.total; o += step) {
        int64_t t = o;
        const int n = (int)(t % a.wo); t /= a.wo;
        const int m = (int)(t % a.ho); t /= a.ho;
        const int j = (int)(t % a.k);
        const int64_t i = t / a.k;
        const int64_t xi = i * a.c * a.h * a.w_in;
        const int64_t wj = (int64_t)j * a.c * a.fh * a.fw;
        float acc = 0.0f;
        for (int r = 0; r < a.c; ++r) {
            for (int u = 0; u < a.fh; ++u) {
                const int64_t yy = (int64_t)m * a.sh + u - a.ph;
                if (yy < 0 || yy >= a.h) continue;
                const int64_t xrow = xi + ((int64_t)r * a.h + yy) * a.w_in;
                const int64_t wrow = wj + ((int64_t)r * a.fh + u) * a.fw;
                for (int v = 0; v < a.fw; ++v) {
                    const int64_t xx = (int64_t)n * a.sw + v - a.pw;
                    if (xx < 0 || xx >= a.w_in) continue;
                    acc = fmaf(load_f(x, xrow + xx), load_f(w, wrow + v), acc);
                }
            }
        }
        a.y[o] = acc;
    }
}

}  // namespace

int launch_direct_conv(const Geometry& g, const void* x, const void* w, float* y,
                       hipStream_t stream, char* err, size_t errlen) {
    DirectArgs a;
    a.x = x;
    a.w = w;
    a.y = y;
    a.total = g.npix * g.k;
    a.c = (int)g.c; a.h = (int)g.h; a.w_in = (int)g.w; a.k = (int)g.k;
    a.fh = (int)g.fh; a.fw = (int)g.fw; a.sh = (int)g.sh; a.sw = (int)g.sw;
    a.ph = (int)g.ph; a.pw = (int)g.pw; a.ho = (int)g.ho; a.wo = (int)g.wo;
    // a grid-stride loop covers any size; 2^20 workgroups are plenty to fill the chip
    const int64_t blocks = std::min<int64_t>((a.total + 255) / 256, int64_t(1) << 20);
    if (g.elem == 4)
        hipLaunchKernelGGL(direct_conv_kernel<float>, dim3((unsigned)blocks), dim3(256), 0, stream, a);
    else
        hipLaunchKernelGGL(direct_conv_kernel<uint16_t>, dim3((unsigned)blocks), dim3(256), 0, stream, a);
    (void)err;
    (void)errlen;
    return 0;
}

}  // namespace im2win
