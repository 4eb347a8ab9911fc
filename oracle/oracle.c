/*
 * CPU oracle for the im2win transform and the im2win-based convolution
 * (Lu, Chu, Liu, "Im2win: Memory Efficient Convolution On SIMD Architectures",
 * arXiv 2306.14320).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path links, loads or calls
 * this file: only the tests, the smoke check and the CPU-baseline leg of the
 * benchmark do.  It shares no code, header or table with the HIP library.
 *
 * Plain, slow, obviously correct: every function is the definition written out
 * as loops, in fp64 for floating point, with no blocking, fusion or reordering.
 * OpenMP only splits independent outputs across threads; it never changes the
 * order of any sum.
 *
 * Shape vector `shp` (int64[11]):
 *   [0] N  [1] C  [2] H  [3] W      input  N x C x H x W   (NCHW, contiguous)
 *   [4] K  [5] Fh [6] Fw            filter K x C x Fh x Fw (contiguous)
 *   [7] sh [8] sw                   stride (rows, columns)
 *   [9] ph [10] pw                  symmetric zero padding (rows, columns)
 *
 * Readings of the paper used here (the paper has no padding and one stride s):
 *   - Output extent is floor((in + 2*pad - f) / s) + 1 (Alg. 1 computes
 *     (Hi - Hf)/s + 1; Table 1, Conv4 maps 224 with a 7-tap filter at stride 2
 *     to 109, so the division is a floor).
 *   - Padding is zeros around the input, as in PyTorch's conv2d; in the window
 *     tensor it appears as +0.0 and a row has Wp = W + 2*pw columns.
 *   - The window for output column n starts at input column n*sw, i.e. at
 *     offset n*sw*Fh of the window-tensor row (Alg. 2 prints n*s*Wf, which
 *     equals this only for square filters).
 */
#include <stdint.h>
#include <string.h>
#include <stddef.h>

#define N_  shp[0]
#define C_  shp[1]
#define H_  shp[2]
#define W_  shp[3]
#define K_  shp[4]
#define FH_ shp[5]
#define FW_ shp[6]
#define SH_ shp[7]
#define SW_ shp[8]
#define PH_ shp[9]
#define PW_ shp[10]

/* Output extent along one axis (Alg. 1, first step; floor per Table 1). */
int64_t oracle_out_extent(int64_t in, int64_t f, int64_t s, int64_t pad) {
    int64_t span = in + 2 * pad - f;
    if (in <= 0 || f <= 0 || s <= 0 || pad < 0 || span < 0) return 0;
    return span / s + 1;
}

/* Columns per window-tensor row.  trimmed = 0: the padded width Wp, every
 * column of the padded input (Sec. III-A sizes the rows with the input width).
 * trimmed = 1: only the columns some window reads; the last window starts at
 * column (Wo-1)*sw and spans Fw columns, so (Wo-1)*sw + Fw. */
int64_t oracle_row_width(const int64_t *shp, int trimmed) {
    if (!trimmed) return W_ + 2 * PW_;
    return (oracle_out_extent(W_, FW_, SW_, PW_) - 1) * SW_ + FW_;
}

/* Elements of the window tensor: N x C x Ho x (Wr * Fh)  (Sec. III-A, size
 * analysis, with the row width Wr in place of Wi). */
int64_t oracle_im2win_elems(const int64_t *shp, int trimmed) {
    int64_t ho = oracle_out_extent(H_, FH_, SH_, PH_);
    return N_ * C_ * ho * oracle_row_width(shp, trimmed) * FH_;
}

/* Elements of the im2col matrix for the same convolution: per image a
 * (Ho*Wo) x (C*Fh*Fw) matrix (Sec. II-B), times N images. */
int64_t oracle_im2col_elems(const int64_t *shp) {
    int64_t ho = oracle_out_extent(H_, FH_, SH_, PH_);
    int64_t wo = oracle_out_extent(W_, FW_, SW_, PW_);
    return N_ * (C_ * FH_ * FW_) * (ho * wo);
}

/* The im2win transformation (Sec. III-A, Eq. 2 read through the copy
 * relation of Alg. 1) with zero padding, written as the value of each element
 * of the window tensor, computed from its flat index e:
 *   e = (((i*C + r)*Ho + m)*Wr + k)*Fh + u   (u fastest: a row holds the Fh
 *                                            input rows column by column)
 *   win[e] = Ipad[i][r][m*sh + u][k],  k < Wr, u < Fh,
 * where Ipad is the input with ph zero rows and pw zero columns on each side.
 * A pure copy of `elem_bytes`-sized elements (4 for fp32, 2 for bf16, 8 for
 * fp64), so the result is unique and any implementation must reproduce it bit
 * for bit. */
void oracle_im2win(const int64_t *shp, const void *x, void *win, int elem_bytes, int trimmed) {
    const int64_t ho = oracle_out_extent(H_, FH_, SH_, PH_);
    const int64_t wr = oracle_row_width(shp, trimmed);
    const int64_t total = N_ * C_ * ho * wr * FH_;
    const unsigned char *src = (const unsigned char *)x;
    unsigned char *dst = (unsigned char *)win;
    const size_t eb = (size_t)elem_bytes;
#pragma omp parallel for
    for (int64_t e = 0; e < total; ++e) {
        const int64_t u = e % FH_;
        const int64_t k = (e / FH_) % wr;
        const int64_t m = (e / (FH_ * wr)) % ho;
        const int64_t plane = e / (FH_ * wr * ho);     /* i*C + r */
        const int64_t yy = m * SH_ + u - PH_;          /* row in the unpadded input */
        const int64_t xx = k - PW_;                    /* column in the unpadded input */
        if (yy >= 0 && yy < H_ && xx >= 0 && xx < W_)
            memcpy(dst + (size_t)e * eb, src + (size_t)((plane * H_ + yy) * W_ + xx) * eb, eb);
        else
            memset(dst + (size_t)e * eb, 0, eb);
    }
}

/* One output of the convolution, Eq. 1 with padding:
 *   O[i][j][m][n] = sum_r sum_u sum_v I[i][r][m*sh+u-ph][n*sw+v-pw] * F[j][r][u][v]
 * summed in fp64 in the order r, u, v.  Out-of-range input positions are the
 * zero padding and contribute nothing.  *abs_out (if non-NULL) receives the sum
 * of |I * F| over the same terms, which bounds the rounding error of any
 * floating-point evaluation of the sum. */
static void conv_one(const int64_t *shp, const double *x, const double *w,
                     int64_t i, int64_t j, int64_t m, int64_t n,
                     double *out, double *abs_out) {
    double acc = 0.0, aacc = 0.0;
    for (int64_t r = 0; r < C_; ++r)
        for (int64_t u = 0; u < FH_; ++u)
            for (int64_t v = 0; v < FW_; ++v) {
                int64_t yy = m * SH_ + u - PH_;
                int64_t xx = n * SW_ + v - PW_;
                if (yy < 0 || yy >= H_ || xx < 0 || xx >= W_) continue;
                double prod = x[((i * C_ + r) * H_ + yy) * W_ + xx]
                            * w[((j * C_ + r) * FH_ + u) * FW_ + v];
                acc += prod;
                aacc += (prod < 0.0) ? -prod : prod;
            }
    *out = acc;
    if (abs_out) *abs_out = aacc;
}

/* Naive direct convolution (Sec. II-C): seven nested loops over the output and
 * the filter.  y is N x K x Ho x Wo; yabs (optional) gets sum |x*w| per output. */
void oracle_direct_conv(const int64_t *shp, const double *x, const double *w,
                        double *y, double *yabs) {
    const int64_t ho = oracle_out_extent(H_, FH_, SH_, PH_);
    const int64_t wo = oracle_out_extent(W_, FW_, SW_, PW_);
#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int64_t i = 0; i < N_; ++i)
        for (int64_t j = 0; j < K_; ++j)
            for (int64_t m = 0; m < ho; ++m)
                for (int64_t n = 0; n < wo; ++n) {
                    int64_t o = ((i * K_ + j) * ho + m) * wo + n;
                    conv_one(shp, x, w, i, j, m, n, &y[o], yabs ? &yabs[o] : NULL);
                }
}

/* The same convolution evaluated only at the given flat NCHW output indices. */
void oracle_direct_conv_at(const int64_t *shp, const double *x, const double *w,
                           const int64_t *idx, int64_t count, double *y, double *yabs) {
    const int64_t ho = oracle_out_extent(H_, FH_, SH_, PH_);
    const int64_t wo = oracle_out_extent(W_, FW_, SW_, PW_);
#pragma omp parallel for schedule(dynamic)
    for (int64_t t = 0; t < count; ++t) {
        int64_t o = idx[t];
        int64_t n = o % wo, m = (o / wo) % ho, j = (o / (wo * ho)) % K_, i = o / (wo * ho * K_);
        conv_one(shp, x, w, i, j, m, n, &y[t], yabs ? &yabs[t] : NULL);
    }
}

/* The im2win-based convolution (Alg. 2's definition of an output) evaluated
 * on a window tensor `win` (N x C x Ho x Wr*Fh, as the transformation writes
 * it), each output computed from its flat NCHW index o = ((i*K + j)*Ho + m)*Wo + n:
 *   O[i][j][m][n] = sum_r sum_u sum_v win[i][r][m][(n*sw + v)*Fh + u] * F[j][r][u][v]
 * summed in fp64 in the order r, u, v.  The window of output column n begins
 * at input column n*sw, which sits at offset n*sw*Fh of the row. */
void oracle_window_conv(const int64_t *shp, const double *win, const double *w, double *y,
                        int trimmed) {
    const int64_t ho = oracle_out_extent(H_, FH_, SH_, PH_);
    const int64_t wo = oracle_out_extent(W_, FW_, SW_, PW_);
    const int64_t row = oracle_row_width(shp, trimmed) * FH_;
    const int64_t total = N_ * K_ * ho * wo;
#pragma omp parallel for schedule(dynamic, 64)
    for (int64_t o = 0; o < total; ++o) {
        const int64_t n = o % wo;
        const int64_t m = (o / wo) % ho;
        const int64_t j = (o / (wo * ho)) % K_;
        const int64_t i = o / (wo * ho * K_);
        double acc = 0.0;
        for (int64_t r = 0; r < C_; ++r)
            for (int64_t u = 0; u < FH_; ++u)
                for (int64_t v = 0; v < FW_; ++v)
                    acc += win[((i * C_ + r) * ho + m) * row + (n * SW_ + v) * FH_ + u]
                         * w[((j * C_ + r) * FH_ + u) * FW_ + v];
        y[o] = acc;
    }
}

/* Brute-force im2col (Sec. II-B): for each image a (Ho*Wo) x (C*Fh*Fw) matrix
 *   M[m*Wo + n][(r*Fh + u)*Fw + v] = Ipad[r][m*sh + u][n*sw + v].
 * cols is N x (Ho*Wo) x (C*Fh*Fw). */
void oracle_im2col(const int64_t *shp, const double *x, double *cols) {
    const int64_t ho = oracle_out_extent(H_, FH_, SH_, PH_);
    const int64_t wo = oracle_out_extent(W_, FW_, SW_, PW_);
    const int64_t kd = C_ * FH_ * FW_;
#pragma omp parallel for
    for (int64_t i = 0; i < N_; ++i)
        for (int64_t m = 0; m < ho; ++m)
            for (int64_t n = 0; n < wo; ++n)
                for (int64_t r = 0; r < C_; ++r)
                    for (int64_t u = 0; u < FH_; ++u)
                        for (int64_t v = 0; v < FW_; ++v) {
                            int64_t yy = m * SH_ + u - PH_;
                            int64_t xx = n * SW_ + v - PW_;
                            double val = 0.0;
                            if (yy >= 0 && yy < H_ && xx >= 0 && xx < W_)
                                val = x[((i * C_ + r) * H_ + yy) * W_ + xx];
                            cols[(i * ho * wo + m * wo + n) * kd + (r * FH_ + u) * FW_ + v] = val;
                        }
}
