// C ABI of libim2win (declared in include/im2win.h): argument validation on
// the host, problem geometry, and kernel dispatch.  Every check runs before
// the first HIP call, so a rejected call enqueues nothing.
#include "im2win.h"
#include "im2win_baseline.h"

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>

#include "common.h"
#include "direct.h"

// Filter scratch of im2win_conv2d_fused_noalloc: a static device array, so
// that the call allocates nothing.  Each device holds its own copy; its
// device address is looked up once per device (with that device current)
// and kept.  Host code uses only that address, never the array's name.
static __device__ __align__(256) unsigned char scratch[IM2WIN_NOALLOC_SCRATCH_BYTES];

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return code;
}

int ok() {
    g_err[0] = '\0';
    return IM2WIN_OK;
}

constexpr int64_t kI31 = (int64_t(1) << 31) - 1;   // kernels index with 32-bit ints
constexpr int64_t kI62 = int64_t(1) << 62;

// a*b with a, b >= 0; returns false if the product exceeds `limit`.
bool mul_le(int64_t a, int64_t b, int64_t limit, int64_t* out) {
    if (a != 0 && b > limit / a) return false;
    *out = a * b;
    return *out <= limit;
}

int geometry(const im2win_desc* d, im2win::Geometry* g) {
    if (!d) return fail(IM2WIN_ENULL, "descriptor is NULL");
    if (d->n < 1 || d->c < 1 || d->h < 1 || d->w < 1 || d->k < 1 || d->fh < 1 || d->fw < 1)
        return fail(IM2WIN_EINVAL,
                    "every size must be >= 1 (n=%lld c=%lld h=%lld w=%lld k=%lld fh=%lld fw=%lld)",
                    (long long)d->n, (long long)d->c, (long long)d->h, (long long)d->w,
                    (long long)d->k, (long long)d->fh, (long long)d->fw);
    if (d->stride_h < 1 || d->stride_w < 1)
        return fail(IM2WIN_EINVAL, "strides must be >= 1 (got %lld, %lld)", (long long)d->stride_h,
                    (long long)d->stride_w);
    if (d->pad_h < 0 || d->pad_w < 0)
        return fail(IM2WIN_EINVAL, "paddings must be >= 0 (got %lld, %lld)", (long long)d->pad_h,
                    (long long)d->pad_w);
    if (d->dtype != IM2WIN_F32 && d->dtype != IM2WIN_BF16)
        return fail(IM2WIN_EINVAL, "unknown dtype %d", (int)d->dtype);
    if (d->layout != IM2WIN_ROWS_PADDED && d->layout != IM2WIN_ROWS_TRIMMED)
        return fail(IM2WIN_EINVAL, "unknown window-tensor layout %d", (int)d->layout);
    const int64_t lim = int64_t(1) << 30;
    if (d->n > kI31 || d->c > lim || d->h > lim || d->w > lim || d->k > lim || d->fh > lim ||
        d->fw > lim || d->stride_h > lim || d->stride_w > lim || d->pad_h > lim || d->pad_w > lim)
        return fail(IM2WIN_EOVERFLOW, "a size, stride or padding exceeds 2^30");
    const int64_t hp = d->h + 2 * d->pad_h, wp = d->w + 2 * d->pad_w;
    if (hp < d->fh || wp < d->fw)
        return fail(IM2WIN_EINVAL,
                    "filter %lldx%lld is larger than the padded input %lldx%lld (Ho or Wo < 1)",
                    (long long)d->fh, (long long)d->fw, (long long)hp, (long long)wp);
    g->n = d->n; g->c = d->c; g->h = d->h; g->w = d->w; g->k = d->k;
    g->fh = d->fh; g->fw = d->fw; g->sh = d->stride_h; g->sw = d->stride_w;
    g->ph = d->pad_h; g->pw = d->pad_w;
    g->ho = (hp - d->fh) / d->stride_h + 1;
    g->wo = (wp - d->fw) / d->stride_w + 1;
    // row width of the window tensor: every padded column, or only those
    // some window reads ((Wo-1)*sw + Fw <= Wp)
    g->wp = d->layout == IM2WIN_ROWS_TRIMMED ? (g->wo - 1) * d->stride_w + d->fw : wp;
    g->elem = d->dtype == IM2WIN_F32 ? 4 : 2;

    // Quantities the kernels hold in 32-bit integers, and element counts.
    int64_t t, t2;
    if (!mul_le(g->wp, d->fh, kI31 / 2, &g->row_len) || !mul_le(g->ho, g->row_len, kI31, &t) ||
        !mul_le(d->fh, d->fw, kI31, &g->taps) || !mul_le(d->h, d->w, kI31, &t) ||
        !mul_le(d->k * 1, d->c, kI31, &t) || !mul_le(t, g->taps, kI31, &t2) ||
        !mul_le(g->ho, g->wo, kI31, &t) || !mul_le(d->n, t, kI31, &g->npix))
        return fail(IM2WIN_EOVERFLOW,
                    "problem too large for 32-bit kernel indexing (N*Ho*Wo, Ho*Wp*Fh, H*W and "
                    "K*C*Fh*Fw must each stay below 2^31)");
    g->used_len = ((g->wo - 1) * g->sw + g->fw) * g->fh;
    return IM2WIN_OK;
}

int bytes_of(const im2win::Geometry& g, int64_t a, int64_t b, int64_t c, int64_t d, size_t* out) {
    int64_t t1, t2, t3, t4;
    if (!mul_le(a, b, kI62, &t1) || !mul_le(t1, c, kI62, &t2) || !mul_le(t2, d, kI62, &t3) ||
        !mul_le(t3, g.elem, kI62, &t4))
        return fail(IM2WIN_EOVERFLOW, "byte size overflows");
    *out = (size_t)t4;
    return IM2WIN_OK;
}

int ws_bytes_of(const im2win::Geometry& g, size_t* out) {
    return bytes_of(g, g.n, g.c, g.ho, g.row_len, out);
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int check_ptr(const void* p, const char* name) {
    if (!p) return fail(IM2WIN_ENULL, "%s is NULL", name);
    if (!aligned16(p)) return fail(IM2WIN_EALIGN, "%s (%p) is not 16-byte aligned", name, p);
    return IM2WIN_OK;
}

// rc: 0, or the IM2WIN_E* code of a failure the launcher detected (msg says which)
int after_launch(int rc, const char* what, const char* msg) {
    if (rc != 0) return fail(rc == IM2WIN_EHIP ? IM2WIN_EHIP : IM2WIN_EOVERFLOW, "%s", msg);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(IM2WIN_EHIP, "%s launch failed: %s", what, hipGetErrorString(e));
    return ok();
}

}  // namespace

extern "C" {

int im2win_workspace_bytes(const im2win_desc* d, size_t* bytes) {
    im2win::Geometry g;
    int rc = geometry(d, &g);
    if (rc) return rc;
    if (!bytes) return fail(IM2WIN_ENULL, "bytes is NULL");
    rc = ws_bytes_of(g, bytes);
    return rc ? rc : ok();
}

int im2win_im2col_bytes(const im2win_desc* d, size_t* bytes) {
    im2win::Geometry g;
    int rc = geometry(d, &g);
    if (rc) return rc;
    if (!bytes) return fail(IM2WIN_ENULL, "bytes is NULL");
    rc = bytes_of(g, g.n, g.ho * g.wo, g.c, g.taps, bytes);
    return rc ? rc : ok();
}

int im2win_output_shape(const im2win_desc* d, int64_t* ho, int64_t* wo) {
    im2win::Geometry g;
    int rc = geometry(d, &g);
    if (rc) return rc;
    if (!ho || !wo) return fail(IM2WIN_ENULL, "ho or wo is NULL");
    *ho = g.ho;
    *wo = g.wo;
    return ok();
}

int im2win_transform(const im2win_desc* d, const void* x, void* ws, size_t ws_bytes, void* stream) {
    im2win::Geometry g;
    int rc = geometry(d, &g);
    if (rc) return rc;
    if ((rc = check_ptr(x, "x")) || (rc = check_ptr(ws, "ws"))) return rc;
    size_t need;
    if ((rc = ws_bytes_of(g, &need))) return rc;
    if (ws_bytes < need)
        return fail(IM2WIN_EWORKSPACE, "workspace holds %zu bytes, the window tensor needs %zu",
                    ws_bytes, need);
    char msg[256] = "";
    rc = im2win::launch_transform(g, x, ws, static_cast<hipStream_t>(stream), msg, sizeof msg);
    return after_launch(rc, "transform", msg);
}

int im2win_filter_scratch_bytes(const im2win_desc* d, size_t* bytes) {
    im2win::Geometry g;
    int rc = geometry(d, &g);
    if (rc) return rc;
    if (!bytes) return fail(IM2WIN_ENULL, "bytes is NULL");
    const int64_t a = im2win::conv_scratch_bytes(g, false), b = im2win::conv_scratch_bytes(g, true);
    *bytes = (size_t)std::max<int64_t>(0, std::max(a, b));
    return ok();
}

int im2win_conv_kernel(const im2win_desc* d, int fused, const char** name) {
    im2win::Geometry g;
    int rc = geometry(d, &g);
    if (rc) return rc;
    if (!name) return fail(IM2WIN_ENULL, "name is NULL");
    *name = im2win::conv_kernel_name(g, fused != 0);
    return ok();
}

int im2win_workspace_shape(const im2win_desc* d, int64_t* dims) {
    im2win::Geometry g;
    int rc = geometry(d, &g);
    if (rc) return rc;
    if (!dims) return fail(IM2WIN_ENULL, "dims is NULL");
    dims[0] = g.n;
    dims[1] = g.c;
    dims[2] = g.ho;
    dims[3] = g.row_len;
    return ok();
}

}  // extern "C"

namespace {

// The filter scratch a convolution variant needs: checked against the
// caller's buffer (NULL is accepted when none is needed).
int check_scratch(const im2win::Geometry& g, bool fused, const void* scratch, size_t scratch_bytes) {
    const int64_t need = im2win::conv_scratch_bytes(g, fused);
    if (need <= 0) return IM2WIN_OK;
    int rc = check_ptr(scratch, "scratch");
    if (rc) return rc;
    if (scratch_bytes < (size_t)need)
        return fail(IM2WIN_EWORKSPACE, "filter scratch holds %zu bytes, this convolution needs %lld",
                    scratch_bytes, (long long)need);
    return IM2WIN_OK;
}

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int static_scratch(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(IM2WIN_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices)
        return fail(IM2WIN_EINVAL, "device %d is beyond the %d devices the static scratch serves", dev,
                    kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(IM2WIN_EHIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                        hipGetErrorString(e));
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return IM2WIN_OK;
}

}  // namespace

extern "C" {

int im2win_conv2d(const im2win_desc* d, const void* ws, size_t ws_bytes, const void* w,
                  void* scratch, size_t scratch_bytes, float* y, void* stream) {
    im2win::Geometry g;
    int rc = geometry(d, &g);
    if (rc) return rc;
    if ((rc = check_ptr(ws, "ws")) || (rc = check_ptr(w, "w")) || (rc = check_ptr(y, "y")))
        return rc;
    size_t need;
    if ((rc = ws_bytes_of(g, &need))) return rc;
    if (ws_bytes < need)
        return fail(IM2WIN_EWORKSPACE, "workspace holds %zu bytes, the window tensor needs %zu",
                    ws_bytes, need);
    if ((rc = check_scratch(g, false, scratch, scratch_bytes))) return rc;
    char msg[256] = "";
    hipStream_t s = static_cast<hipStream_t>(stream);
    rc = g.elem == 4 ? im2win::launch_conv_f32(g, false, ws, w, scratch, y, s, msg, sizeof msg)
                     : im2win::launch_conv_bf16(g, false, ws, w, scratch, y, s, msg, sizeof msg);
    return after_launch(rc, "conv2d", msg);
}

int im2win_conv2d_fused(const im2win_desc* d, const void* x, const void* w, void* scratch,
                        size_t scratch_bytes, float* y, void* stream) {
    im2win::Geometry g;
    int rc = geometry(d, &g);
    if (rc) return rc;
    if ((rc = check_ptr(x, "x")) || (rc = check_ptr(w, "w")) || (rc = check_ptr(y, "y")))
        return rc;
    if ((rc = check_scratch(g, true, scratch, scratch_bytes))) return rc;
    char msg[256] = "";
    hipStream_t s = static_cast<hipStream_t>(stream);
    rc = g.elem == 4 ? im2win::launch_conv_f32(g, true, x, w, scratch, y, s, msg, sizeof msg)
                     : im2win::launch_conv_bf16(g, true, x, w, scratch, y, s, msg, sizeof msg);
    return after_launch(rc, "conv2d_fused", msg);
}

int im2win_conv2d_fused_noalloc(const im2win_desc* d, const void* x, const void* w, float* y,
                                void* stream) {
    im2win::Geometry g;
    int rc = geometry(d, &g);
    if (rc) return rc;
    if ((rc = check_ptr(x, "x")) || (rc = check_ptr(w, "w")) || (rc = check_ptr(y, "y")))
        return rc;
    const int64_t need = im2win::conv_scratch_bytes(g, true);
    if (need > (int64_t)IM2WIN_NOALLOC_SCRATCH_BYTES)
        return fail(IM2WIN_EWORKSPACE,
                    "this convolution needs %lld bytes of filter scratch; the library's static "
                    "scratch holds %lld (use im2win_conv2d_fused with a scratch buffer)",
                    (long long)need, (long long)IM2WIN_NOALLOC_SCRATCH_BYTES);
    void* sp = nullptr;
    if (need > 0 && (rc = static_scratch(&sp))) return rc;
    char msg[256] = "";
    hipStream_t s = static_cast<hipStream_t>(stream);
    rc = g.elem == 4 ? im2win::launch_conv_f32(g, true, x, w, sp, y, s, msg, sizeof msg)
                     : im2win::launch_conv_bf16(g, true, x, w, sp, y, s, msg, sizeof msg);
    return after_launch(rc, "conv2d_fused_noalloc", msg);
}

int im2win_direct_conv2d(const im2win_desc* d, const void* x, const void* w, float* y,
                         void* stream) {
    im2win::Geometry g;
    int rc = geometry(d, &g);
    if (rc) return rc;
    if (!x || !w || !y) return fail(IM2WIN_ENULL, "%s is NULL", !x ? "x" : !w ? "w" : "y");
    char msg[256] = "";
    rc = im2win::launch_direct_conv(g, x, w, y, static_cast<hipStream_t>(stream), msg, sizeof msg);
    return after_launch(rc, "direct_conv2d", msg);
}

const char* im2win_last_error(void) { return g_err; }

int im2win_check_plan(const im2win_desc* d) {
    im2win::Geometry g;
    int rc = geometry(d, &g);
    if (rc) return rc;
    char msg[256];
    const int64_t v = im2win::check_plans(g, msg, sizeof msg);
    if (v == 0) return ok();
    fail(0, "%lld plan violation(s); first: %s", (long long)v, msg);
    return v > 0x7fffffff ? 0x7fffffff : (int)v;
}

int im2win_selftest(void) {
    int failures = 0;
    const uint32_t divisors[] = {1, 2, 3, 5, 6, 7, 9, 11, 14, 15, 25, 48, 49, 56, 96, 121, 174,
                                 196, 1603, 1610, 3136, 12544, 65535, 65536, 65537, 1000003,
                                 (1u << 30) - 1, 1u << 30, (1u << 31) - 1};
    for (uint32_t d : divisors) {
        const im2win::FastDiv f = im2win::make_fastdiv(d);
        const uint32_t probes[] = {0u, 1u, d - 1, d, d + 1, 2 * d - 1, 12345u, 999999u,
                                   (1u << 31) - 1, (1u << 31) - 2, (1u << 31) - d};
        for (uint32_t n : probes) {
            if (n >= (1u << 31)) continue;
            if (im2win::fast_div(n, f) != n / d) ++failures;
        }
        // every multiple boundary for the first few thousand quotients
        for (uint32_t q = 0; q < 4096; ++q) {
            const uint64_t base = uint64_t(q) * d;
            for (int64_t delta = -1; delta <= 1; ++delta) {
                const int64_t n = int64_t(base) + delta;
                if (n < 0 || n >= (int64_t(1) << 31)) continue;
                if (im2win::fast_div(uint32_t(n), f) != uint32_t(n) / d) ++failures;
            }
        }
    }
    return failures;
}

}  // extern "C"
