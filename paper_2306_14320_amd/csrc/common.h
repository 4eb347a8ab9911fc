// Internal declarations shared by the HIP translation units of libim2win.
// Not part of the public ABI (that is include/im2win.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace im2win {

// ---------------------------------------------------------------------------
// Division by a launch-invariant divisor, for index decomposition in kernels.
//
// Granlund & Montgomery, "Division by Invariant Integers using
// Multiplication" (PLDI 1994), Sec. 4: with l = ceil(log2 d) and
// m = floor(2^32 * (2^l - d) / d) + 1, floor(n / d) = (mulhi(m, n) + n) >> l
// for every 32-bit n.  We only use numerators below 2^31, so the sum
// mulhi(m, n) + n cannot overflow 32 bits.
// ---------------------------------------------------------------------------
struct FastDiv {
    uint32_t d;
    uint32_t mul;
    uint32_t shift;
};

__host__ __device__ inline FastDiv make_fastdiv(uint32_t d) {
    FastDiv f;
    f.d = d;
    uint32_t l = 0;
    while ((uint64_t(1) << l) < d) ++l;
    f.shift = l;
    f.mul = uint32_t(((uint64_t(1) << 32) * ((uint64_t(1) << l) - d)) / d + 1);
    return f;
}

__host__ __device__ inline uint32_t fast_div(uint32_t n, const FastDiv& f) {
#if defined(__HIP_DEVICE_COMPILE__)
    uint32_t t = __umulhi(n, f.mul);
#else
    uint32_t t = uint32_t((uint64_t(n) * f.mul) >> 32);
#endif
    return (t + n) >> f.shift;
}

// ---------------------------------------------------------------------------
// Problem geometry, derived once on the host from the public descriptor.
// ---------------------------------------------------------------------------
struct Geometry {
    int64_t n, c, h, w, k, fh, fw, sh, sw, ph, pw;
    int64_t ho, wo, wp;
    int64_t row_len;      // L = Wp * Fh, length of one window-tensor row
    int64_t used_len;     // Lu = ((Wo-1)*sw + Fw) * Fh, the part of a row windows read
    int64_t taps;         // T = Fh * Fw
    int64_t npix;         // N * Ho * Wo, the implicit GEMM's pixel dimension
    int elem;             // bytes per element of x / w / window tensor
};

// ---------------------------------------------------------------------------
// Transformation
// ---------------------------------------------------------------------------
struct XformArgs {
    const void* x;
    void* ws;
    int64_t nc;          // N*C image planes
    int h, w, ho, wp, fh, sh, ph, pw;
    int row_len;         // L = Wp*Fh
    int g;               // planes per workgroup (>1 only when tm == ho)
    int tm;              // window-tensor rows per plane per workgroup
    int tiles_per_plane; // ceil(ho / tm)
    int vec;             // elements per 16 bytes
    int vec_in;          // planes and rows of x are whole 16-byte vectors
    FastDiv div_plane, div_w, div_sh;   // by H*W, W, sh
};

// The run of window-tensor rows one workgroup of the LDS kernel produces.
// The workgroup builds the run in LDS (index 0 = global element obase - shift,
// so that 16-byte LDS reads and global stores line up) and copies it out.
struct XformBlock {
    int64_t plane0;   // first image plane (i*C + r)
    int nplanes;      // planes in this workgroup
    int m0, nrows;    // window-tensor rows [m0, m0 + nrows) of each plane
    int y_lo, nrin;   // input rows [y_lo, y_lo + nrin) of each plane that the run uses
    int64_t obase;    // first output element
    int olen;         // output elements (one contiguous run)
    int shift;        // obase mod (16 bytes / element size)

    __host__ __device__ void init(int64_t b, const XformArgs& a) {
        const int64_t grp = b / a.tiles_per_plane;
        const int tile = (int)(b - grp * a.tiles_per_plane);
        plane0 = grp * a.g;
        nplanes = (int)(a.nc - plane0 < a.g ? a.nc - plane0 : a.g);
        m0 = tile * a.tm;
        nrows = a.ho - m0 < a.tm ? a.ho - m0 : a.tm;
        const int lo = m0 * a.sh - a.ph;
        const int hi = (m0 + nrows - 1) * a.sh - a.ph + a.fh;
        y_lo = lo > 0 ? lo : 0;
        const int y_hi = hi < a.h ? hi : a.h;
        nrin = y_hi - y_lo > 0 ? y_hi - y_lo : 0;
        obase = (plane0 * a.ho + m0) * (int64_t)a.row_len;
        olen = nplanes * nrows * a.row_len;
        shift = (int)(obase % a.vec);
    }
    // Window-tensor rows [*m_first, *m_last] of this run that use input row
    // yy (each at row-in-window u = yy + ph - m*sh); empty when first > last.
    __host__ __device__ void rows_of(int yy, const XformArgs& a, int* m_first, int* m_last) const {
        const int t = yy + a.ph;                       // >= 0
        const int hi = (int)fast_div((uint32_t)t, a.div_sh);
        const int lo_num = t - a.fh + a.sh;            // ceil((t - fh + 1) / sh)
        const int lo = lo_num > 0 ? (int)fast_div((uint32_t)lo_num, a.div_sh) : 0;
        *m_first = lo > m0 ? lo : m0;
        *m_last = hi < m0 + nrows - 1 ? hi : m0 + nrows - 1;
    }
    // LDS index of window-tensor element (plane p of the run, row m, column k, u)
    __host__ __device__ int lds_index(int p, int m, int k, int u, const XformArgs& a) const {
        return shift + (p * nrows + (m - m0)) * a.row_len + k * a.fh + u;
    }
};

struct XformPlan {
    bool use_lds = false;     // LDS-staged kernel, else the direct fallback
    int64_t g = 1;            // planes per workgroup
    int64_t tm = 1;           // window-tensor rows per plane per workgroup
    int64_t tiles_per_plane = 1;
    int64_t lds_bytes = 0;
    int64_t blocks = 0;
};

XformPlan plan_transform(const Geometry& g);
XformArgs transform_args(const Geometry& g, const XformPlan& p, const void* x, void* ws);

int launch_transform(const Geometry& g, const void* x, void* ws, hipStream_t stream,
                     char* err, size_t errlen);

// ---------------------------------------------------------------------------
// Convolution kernels.  `fused` selects where the window strips come from:
// false -> the window tensor `src`; true -> the input tensor `src`.
// ---------------------------------------------------------------------------
// `scratch` (device, caller-owned) receives the repacked filter when the
// plan reads one; it holds at least conv_scratch_bytes(g, fused) bytes.
int launch_conv_f32(const Geometry& g, bool fused, const void* src, const void* w, void* scratch,
                    float* y, hipStream_t stream, char* err, size_t errlen);
int launch_conv_bf16(const Geometry& g, bool fused, const void* src, const void* w, void* scratch,
                     float* y, hipStream_t stream, char* err, size_t errlen);

// Bytes of device scratch (the repacked filter) the tiled convolution of
// this geometry needs, 0 when its kernels read w as given; -1 when no tile
// fits in LDS, in which case launch_conv_plain computes the convolution.
int64_t conv_scratch_bytes(const Geometry& g, bool fused);
// Name of the kernel family the convolution launches (static string).
const char* conv_kernel_name(const Geometry& g, bool fused);

// One thread per output, reading the window tensor (or x, fused) and the
// filter straight from device memory: the convolution of any shape whose
// window strips do not fit the tiled kernels' LDS.
int launch_conv_plain(const Geometry& g, bool fused, const void* src, const void* w, float* y,
                      hipStream_t stream, char* err, size_t errlen);

// Host-side bounds check of the launch plans (see im2win_check_plan).
// Returns the number of violations; the first is described in `msg`.
int64_t check_plans(const Geometry& g, char* msg, size_t msglen);

}  // namespace im2win
