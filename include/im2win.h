/*
 * im2win.h -- C ABI of the MI355X (gfx950) im2win transform and im2win-based
 * 2-D convolution.
 *
 * Method: Lu, Chu, Liu, "Im2win: Memory Efficient Convolution On SIMD
 * Architectures" (arXiv 2306.14320).  Sec. II-A defines the convolution
 * (Eq. 1); Sec. III-A and Alg. 1 define the im2win transformation and its
 * size; Alg. 2 defines the convolution that reads the transformed tensor.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Tensors are dense and contiguous (Sec. I: every tensor is a 1-D array in
 *    NCHW order, W fastest):
 *      x  input   N x C x H x W
 *      w  filter  K x C x Fh x Fw
 *      y  output  N x K x Ho x Wo, always fp32
 *      ws window tensor N x C x Ho x (Wr*Fh), same dtype as x
 *    with Wr the row width of d->layout (Wp = W + 2*pad_w by default),
 *         Ho = floor((H + 2*pad_h - Fh) / stride_h) + 1,
 *         Wo = floor((W + 2*pad_w - Fw) / stride_w) + 1.
 *  - Padding is symmetric zero padding (not in the paper; the convolution is
 *    the one of PyTorch's conv2d with these strides and paddings, no bias, no
 *    dilation, no groups).
 *  - Device pointers (x, w, ws, scratch, y) are owned by the caller; the
 *    library never allocates, frees or keeps device memory.  Each pointer
 *    must be 16-byte aligned and the buffers must not overlap.
 *  - `stream` is a hipStream_t (NULL = the legacy default stream).  Calls only
 *    enqueue work: they never synchronise and hold no state between calls,
 *    so they may be made from several host threads at once.  Buffers a call
 *    writes (ws, scratch, y) must not be in use by other work that may run
 *    concurrently with it (another stream, another thread's call): calls on
 *    one stream may share them, since the stream orders them.
 *  - Return value: IM2WIN_OK or a negative IM2WIN_E* code.  Arguments are
 *    validated on the host before any HIP call, so an invalid call enqueues
 *    nothing.  im2win_last_error() then describes the failure.
 *  - Accumulation is fp32 for both dtypes; results are within the fp32
 *    rounding of the exact sum (no bit-exact promise across kernel versions).
 */
#ifndef IM2WIN_H
#define IM2WIN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Element type of x, w and the window tensor.  y is fp32 in both cases. */
typedef enum {
    IM2WIN_F32 = 0,   /* IEEE binary32 */
    IM2WIN_BF16 = 1   /* bfloat16; products and sums in fp32 */
} im2win_dtype;

/*
 * Width Wr of the window tensor's rows, in input columns (each row holds
 * Wr*Fh elements).
 *  - PADDED: Wr = Wp = W + 2*pad_w, every column of the padded input
 *    (Sec. III-A sizes the tensor with the full input width).
 *  - TRIMMED: Wr = Wt = (Wo-1)*stride_w + Fw, only the columns some window
 *    reads (the padded layout also holds the trailing columns the last
 *    window does not reach).  Then the window tensor is never larger than
 *    the im2col matrix when Fw >= stride_w: im2col - im2win =
 *    N*C*Fh*Ho*(Wo-1)*(Fw - stride_w) elements.
 * Both layouts give the same convolution; a window tensor must be read with
 * the layout it was written with.
 */
typedef enum {
    IM2WIN_ROWS_PADDED = 0,
    IM2WIN_ROWS_TRIMMED = 1
} im2win_layout;

/* Problem description (all fields by value, nothing retained). */
typedef struct {
    int64_t n, c, h, w;          /* input N x C x H x W */
    int64_t k, fh, fw;           /* filter K x C x Fh x Fw */
    int64_t stride_h, stride_w;  /* >= 1 */
    int64_t pad_h, pad_w;        /* >= 0, zero padding on both sides */
    int32_t dtype;               /* an im2win_dtype */
    int32_t layout;              /* an im2win_layout; 0 (zero-initialised) = PADDED */
} im2win_desc;

enum {
    IM2WIN_OK = 0,
    IM2WIN_EINVAL = -1,      /* bad shape, stride, padding, dtype, layout, or Ho/Wo < 1 */
    IM2WIN_ENULL = -2,       /* a required pointer is NULL */
    IM2WIN_EWORKSPACE = -3,  /* ws_bytes or scratch_bytes is smaller than the call needs */
    IM2WIN_EHIP = -4,        /* the HIP runtime reported an error at launch */
    IM2WIN_EOVERFLOW = -5,   /* a size exceeds what the kernels index */
    IM2WIN_EALIGN = -6       /* a device pointer is not 16-byte aligned */
};

/*
 * Size in bytes of the window tensor, N*C*Ho*(Wr*Fh)*sizeof(dtype)
 * (Sec. III-A size analysis: N x C x Ho x (Wi*Hf), with the row width Wr of
 * d->layout in place of Wi).  Unlike Alg. 1, which falls back to the input
 * size when Fh <= stride, this is always the full N x C x Ho x Wr*Fh tensor
 * that im2win_transform writes.
 * Host only; `bytes` receives the size.  Errors: EINVAL, ENULL, EOVERFLOW.
 */
int im2win_workspace_bytes(const im2win_desc* d, size_t* bytes);

/*
 * Size in bytes an im2col matrix of the same convolution would take,
 * N*(Ho*Wo)*(C*Fh*Fw)*sizeof(dtype) (Sec. II-B), for comparison with
 * im2win_workspace_bytes().  Host only.  Errors: EINVAL, ENULL, EOVERFLOW.
 */
int im2win_im2col_bytes(const im2win_desc* d, size_t* bytes);

/*
 * Output extents Ho and Wo (Alg. 1, first step, with floor division and
 * padding).  Host only.  Errors: EINVAL, ENULL.
 */
int im2win_output_shape(const im2win_desc* d, int64_t* ho, int64_t* wo);

/*
 * Shape of the window tensor (Sec. III-A: N x C x Ho x (Wi*Hf), with the row
 * width Wr of d->layout in place of Wi): dims[0..3] = N, C, Ho, Wr*Fh, in
 * elements of d->dtype.  Host only; `dims` points to 4 int64_t.
 * Errors: EINVAL, ENULL, EOVERFLOW.
 */
int im2win_workspace_shape(const im2win_desc* d, int64_t* dims);

/*
 * Size in bytes of the filter scratch that im2win_conv2d and
 * im2win_conv2d_fused take for this descriptor (0 when neither needs one).
 * Alg. 3 reads the filter transposed, F[j][r][v][u], so that a filter row
 * follows the window order (v*Fh + u) of the window tensor; the matrix-core
 * kernels go further and copy the filter to on-chip memory in the order of
 * their reduction.  For the shapes where the filter rows are not whole
 * 16-byte vectors in that order (fp32: C*Fh*Fw per tile chunk not a multiple
 * of 4 floats), and for the bf16 kernels that stage 8-channel pieces
 * (C a multiple of 16, K a multiple of the tile, 3x3, 3x5 or 1x1 filters),
 * each convolution call first rewrites w into the scratch in that order and
 * the kernels read it from there.  The size is at most about
 * K*C*Fh*Fw*sizeof(dtype), padded to the kernels' tile.  The same buffer may
 * serve both entry points and every call with this descriptor.
 * Host only.  Errors: EINVAL, ENULL, EOVERFLOW.
 */
int im2win_filter_scratch_bytes(const im2win_desc* d, size_t* bytes);

/*
 * The im2win transformation (Alg. 1, Eq. 2) with zero padding:
 *   ws[i][r][m][k*Fh + u] = x[i][r][m*stride_h + u - pad_h][k - pad_w]
 * for k < Wr, u < Fh, and +0 where the source lies in the padding.  Each row
 * of the window tensor holds, column by column, the Fh input rows that the
 * windows of output row m cover, so the window of output column n is the
 * contiguous run [n*stride_w*Fh, (n*stride_w + Fw)*Fh) of that row.
 * An exact copy: every element of ws (all ws_bytes of the tensor's size) is
 * written, with the bit pattern of its source or +0.
 *   x   device, N x C x H x W, dtype d->dtype (read only)
 *   ws  device, at least im2win_workspace_bytes() bytes (written)
 * Errors: EINVAL, ENULL, EALIGN, EWORKSPACE, EOVERFLOW, EHIP.
 */
int im2win_transform(const im2win_desc* d, const void* x, void* ws, size_t ws_bytes,
                     void* stream);

/*
 * The im2win-based convolution (Alg. 2; Sec. III-B for the data reuse it is
 * built around) reading the window tensor written by im2win_transform:
 *   y[i][j][m][n] = sum_r sum_u sum_v ws[i][r][m][(n*stride_w + v)*Fh + u] * w[j][r][u][v]
 * (Alg. 2 prints the window offset as n*s*Wf; the window of output column n
 * starts at input column n*stride_w, i.e. at n*stride_w*Fh in the row, which
 * is the same for the square filters the paper evaluates.)
 * y is overwritten (not accumulated into).  Products and sums are fp32 on
 * the matrix cores, for both dtypes.  Shapes whose window strips no on-chip
 * tile holds (rows of very many columns with few output columns) run on a
 * kernel with one thread per output instead, with the same definition.
 *   ws       device, the window tensor of x for this descriptor (read only)
 *   w        device, K x C x Fh x Fw, dtype d->dtype (read only)
 *   scratch  device, scratch_bytes >= im2win_filter_scratch_bytes() (written:
 *            the repacked filter); may be NULL when that size is 0
 *   y        device, N x K x Ho x Wo fp32 (written)
 * Errors: EINVAL, ENULL, EALIGN, EWORKSPACE (ws or scratch too small),
 * EOVERFLOW, EHIP.
 */
int im2win_conv2d(const im2win_desc* d, const void* ws, size_t ws_bytes, const void* w,
                  void* scratch, size_t scratch_bytes, float* y, void* stream);

/*
 * The same convolution computed straight from x: each workgroup builds the
 * window-tensor rows it needs in on-chip memory (LDS) and never writes the
 * window tensor to device memory, so no workspace is needed.  Same result
 * definition, accumulation and output as im2win_conv2d.
 *   x        device, N x C x H x W (read only); w, scratch, y as above
 * Errors: EINVAL, ENULL, EALIGN, EWORKSPACE (scratch too small), EOVERFLOW,
 * EHIP.
 */
int im2win_conv2d_fused(const im2win_desc* d, const void* x, const void* w, void* scratch,
                        size_t scratch_bytes, float* y, void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * convolution as im2win_conv2d_fused with no scratch argument.  The repacked
 * filter goes to a static device array of IM2WIN_NOALLOC_SCRATCH_BYTES inside
 * the library, one per device, held until the process ends; the call
 * allocates and frees nothing.  The device current on the calling thread
 * must be the device of x, w, y and the stream.
 * Every call on a device shares that device's array: calls that may overlap
 * on one device (other streams, other host threads) race on it and must be
 * serialised by the caller; calls on one stream are ordered and safe.  Each
 * call rewrites the part of the array it reads before reading it.
 *   x, w, y  as for im2win_conv2d_fused
 * Errors: EINVAL, ENULL, EALIGN, EOVERFLOW, EHIP, and EWORKSPACE when
 * im2win_filter_scratch_bytes() exceeds IM2WIN_NOALLOC_SCRATCH_BYTES (use
 * im2win_conv2d_fused with a caller buffer then).
 */
#define IM2WIN_NOALLOC_SCRATCH_BYTES (8u << 20)
int im2win_conv2d_fused_noalloc(const im2win_desc* d, const void* x, const void* w, float* y,
                                void* stream);

/*
 * Name of the convolution kernel that im2win_conv2d (fused == 0) or
 * im2win_conv2d_fused (fused != 0) launches for *d, for logs, profiles and
 * tests.  *name receives a string owned by the library (valid for the life of
 * the process), one of:
 *   "f32_bands"          fp32, a band of output rows of one image (or of
 *                        several whole small images) x 32 or 64 output
 *                        channels per workgroup
 *   "f32_bands_small_c"  fp32 with 3 input channels and a 3x3, 7x7 or 11x11
 *                        filter: runs of bands of rows x 64 output channels
 *                        per workgroup, each band's whole reduction staged
 *                        at once
 *   "f32_tiles"          fp32, tiles of output channels x pixels
 *   "bf16_one_image"     bf16, one image x 128 output channels per workgroup
 *   "bf16_tiles"         bf16, tiles of output channels x pixels
 *   "bf16_widened_tiles" bf16 inputs widened to fp32 in the fp32 tile kernel
 *   "per_output"         one thread per output (no tile fits on chip)
 * Host only.  Errors: EINVAL, ENULL, EOVERFLOW.
 */
int im2win_conv_kernel(const im2win_desc* d, int fused, const char** name);

/*
 * Message for the last failed call on this host thread ("" if none).  The
 * string is owned by the library and valid until the next call on the thread.
 */
const char* im2win_last_error(void);

/*
 * Host-side self check of the library's integer arithmetic helpers (division
 * by invariant divisors used for index decomposition).  Returns 0 when every
 * check passes, otherwise the number of failures.  No HIP calls.
 */
int im2win_selftest(void);

/*
 * Host-side check of the launch plan the library would use for *d: replays
 * every workgroup of the transformation and of both convolutions with the
 * kernels' own index arithmetic and verifies that every LDS and device-memory
 * index stays inside its buffer and that the workgroups cover each output
 * exactly once.  Returns 0 when all checks pass, the number of violations
 * (> 0, first one in im2win_last_error()) otherwise, or a negative IM2WIN_E*
 * code for an invalid descriptor.  No HIP calls; cost grows with the size of
 * the problem (it visits every window-tensor element once).
 */
int im2win_check_plan(const im2win_desc* d);

#ifdef __cplusplus
}
#endif

#endif /* IM2WIN_H */
