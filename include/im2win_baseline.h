/*
 * im2win_baseline.h -- comparison baseline exported by libim2win beside the
 * im2win entry points of im2win.h (same descriptor, error codes and
 * conventions; see there).
 *
 * The paper measures its im2win convolution against an im2col-based
 * convolution and against a direct convolution that transforms nothing
 * (Sec. IV-B, Fig. 4).  The im2col baseline is the framework's own unfold and
 * GEMM; the direct one is this entry point.  The im2win path never calls it.
 */
#ifndef IM2WIN_BASELINE_H
#define IM2WIN_BASELINE_H

#include "im2win.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * y = the convolution of Eq. 1 computed directly from x and w, with no data
 * transformation and no workspace: one GPU thread per output element sums
 * x * w over channel, filter row and filter column (in that order, fp32
 * fused multiply-adds; bf16 operands are widened exactly).  Input and filter
 * are read straight from global memory, so this is the plain direct
 * convolution, not a tuned kernel.
 *   x  device, N x C x H x W, dtype d->dtype (read only)
 *   w  device, K x C x Fh x Fw, dtype d->dtype (read only)
 *   y  device, N x K x Ho x Wo fp32, fully overwritten
 * Pointers need only the alignment of their element type.  Asynchronous on
 * `stream`; holds no state.  Errors: EINVAL, ENULL, EOVERFLOW (as
 * im2win_conv2d_fused), EHIP.
 */
int im2win_direct_conv2d(const im2win_desc* d, const void* x, const void* w, float* y,
                         void* stream);

#ifdef __cplusplus
}
#endif

#endif /* IM2WIN_BASELINE_H */
