// Comparison baseline of libim2win (exported as im2win_direct_conv2d):
// direct convolution with no data transformation.  Internal declaration.
#pragma once

#include "common.h"

namespace im2win {

int launch_direct_conv(const Geometry& g, const void* x, const void* w, float* y,
                       hipStream_t stream, char* err, size_t errlen);

}  // namespace im2win
